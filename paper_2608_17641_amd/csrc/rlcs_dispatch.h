// Host-side pieces shared by the entry points: argument checks (all before any HIP call),
// the choice of kernel variant, and the launches. Each entry point lives in its own
// translation unit so that the library's kernels compile in parallel.
#pragma once

#include <hip/hip_runtime.h>

#include <atomic>
#include <climits>
#include <cstdint>
#include <initializer_list>
#include <type_traits>

#include "rlcs.h"
#include "rlcs_kernels.h"

namespace rlcs {
namespace host {

// Workgroups of `kernel` (with `threads` lanes) that the current device holds at once, or 0.
template <class Kernel>
int64_t resident_groups(Kernel kernel, int threads) {
    int dev = 0, cus = 0, per_cu = 0;
    if (hipGetDevice(&dev) != hipSuccess) return 0;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kernel, threads, 0) != hipSuccess) return 0;
    return int64_t(cus) * per_cu;
}

// Waves per workgroup: 4 for rows of up to 4*64*K steps (several rows per workgroup), 16 for
// longer rows (one row, or a 16*64*K-step tile of one, per workgroup).
constexpr int kSmallWaves = 4;
constexpr int kLargeWaves = 16;
// Rows of 32*K to 64*K steps (at most two rows per wave, whole rows per wave) run one-wave
// workgroups for the policies where that measured faster (C harness, cold: 4096 x 256 fp32 GAE
// 5.76 -> 5.68 us, eligibility traces 3.45 -> 3.38 us, bf16 GAE 16384 x 512 25.6 -> 25.1 us);
// V-Trace, Retrace and TD(lambda) ran 2-7 % slower so and keep four-wave workgroups.
// Wave-rows calls of float32 GAE with truncation take workgroups of four waves (each wave still
// on its own) from 2^18 to 2^20 steps (1024 to 4096 waves), one wave per workgroup otherwise.
// Measured (C harness, cold, one-wave against four-wave workgroups): 4096 x 256 5.21 -> 4.78 us,
// 8192 x 128 5.20 -> 4.85, 16384 x 64 5.23 -> 4.91, 4096 x 128 3.55 -> 3.49, 2048 x 256 3.53 ->
// 3.49, 1024 x 256 3.00 -> 2.92; with fewer waves the four-wave grid leaves CUs idle (512 x 256
// 2.57 -> 2.59, 4096 x 32 2.59 -> 2.70); above 2^20 steps four waves lose 4-8 % (6144 x 256 6.17
// -> 6.68, 16384 x 256 14.6 -> 15.3), and so they do without truncation (4096 x 256 4.29 ->
// 4.46), for bfloat16 (16384 x 64 4.69 -> 4.92) and for V-Trace (4096 x 256 6.03 -> 6.16). Two
// waves per workgroup lost everywhere, eight gained less than four.
constexpr int64_t kWaveRowsQuadMinSteps = int64_t(1) << 18;
constexpr int64_t kWaveRowsQuadSteps = int64_t(1) << 20;
template <class Op, typename DT, bool TR> struct WaveRowsQuads : std::false_type {};
template <> struct WaveRowsQuads<GaeOp, float, true> : std::true_type {};

template <class Op> struct OneWaveRows : std::false_type {};
template <> struct OneWaveRows<GaeOp> : std::true_type {};
template <bool D, bool S> struct OneWaveRows<ForwardOp<D, S>> : std::true_type {};

// Staged policies (full-form Retrace) use 4 waves when a 4-wave chunk's slices fit in 64 KB of
// LDS, else 2 waves when two 2-wave workgroups fit in a CU's 160 KB (80 KB each; 4096 x 256 x 18
// fp32 49.6 -> 48.5 us against one wave), else 1 wave.
constexpr int kStagedWaves = 1;
constexpr int kStagedMidWaves = 2;
constexpr int64_t kStagedLdsBudget = 64 * 1024;
constexpr int64_t kStagedMidLdsBudget = 80 * 1024;
// LDS of a sliced chunk (long action axes, one wave): room for slices of one whole 128-byte line
// of float32 actions (two slabs of 257 x 32 elements, 65.8 KB), two workgroups per CU.
constexpr int64_t kSlicedLdsBudget = 80 * 1024;

// Steps per lane: one 16-byte vector of each input.
template <typename DT> struct Width;
template <> struct Width<float> { static constexpr int K = 4; };
template <> struct Width<bf16_t> { static constexpr int K = 8; };

// Smallest tile of the split-row variant (float32, 4 waves), which sizes the workspace.
constexpr int64_t kMinTile = int64_t(kSmallWaves) * kWave * Width<float>::K;

// Rows longer than one large workgroup's chunk are split across workgroups (a workspace given,
// T a multiple of K) when there are fewer than kSplitBelowRows of them. With more rows, or
// shorter ones, whole-row workgroups are faster: a tile waiting for its neighbours' maps costs
// more than the idle CUs (timed: 64 x 4096 fp32 GAE 3.9 us whole-row, 5.2 us split; 512 x 8192
// the same either way; 16 x 16384 bf16 9.2 us whole-row, 6.4 us split).
constexpr int64_t kSplitBelowRows = 256;
// Split rows use 4-wave tiles, or 16-wave tiles when a row would have more than this many
// 4-wave ones (all tiles of a row draw their tickets from one word).
constexpr int64_t kMaxSmallTilesPerRow = 64;

// Largest action axis of full-form Retrace whose chunk's whole [steps, A] slices are staged in
// LDS; longer axes are staged in slices of sliced_width actions.
constexpr int64_t kMaxActions = 28;

// Longest supported row (the kernels keep offsets within a row range in 32 bits).
constexpr int64_t kMaxT = int64_t(1) << 30;

// Kernel-variant override of the calling thread (rlcs_testing_set_variant, a test-only entry
// point); defined in rlcs_common.hip.
extern thread_local int g_variant;

inline bool aligned(const void* p, size_t a) { return reinterpret_cast<uintptr_t>(p) % a == 0; }
inline bool unit_interval(float x) { return x >= 0.f && x <= 1.f; }  // false for NaN
inline bool positive(float x) { return x > 0.f; }                     // false for NaN, true for +inf

inline size_t dtype_size(rlcs_dtype d) { return d == RLCS_BF16 ? 2 : 4; }

// Common checks of sizes, dtype and the element alignment of every given pointer.
inline rlcs_status check_common(int64_t N, int64_t T, rlcs_dtype dtype,
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
    int64_t tiles_per_row;  // tiles kernel: tiles of each row (grid = N * tiles_per_row)
    int64_t rows_per_wg;  // rows kernel: rows per workgroup
    int wave_local;       // rows kernel: no carry crosses waves
    size_t lds_bytes;     // dynamic LDS (staged policies)
    bool pad;             // rows kernel, vector path: lanes outside the range or in row gaps skip
    int wave_rows_log2T;  // >= 0: wave_rows_kernel (rows tile a wave exactly; T = 2^log2T)
    int flat_R;           // > 0: flat_rows_kernel with this many whole rows per workgroup
    int flat_W;           // its waves per workgroup (4, or 16 for float32 rows)
    uint32_t flat_magic;  // ceil(2^flat_shift(flat_W) / T): a lane's row by multiply-shift
};

template <class Op, typename DT, bool VEC, bool TR, int W, bool PAD = false>
void launch_w(const Args& a, const Plan& p, hipStream_t stream) {
    constexpr int K = Width<DT>::K;
    const dim3 block(W * kWave);
    if constexpr (Op::kStaged == 0) {
        if (p.split) {
            hipLaunchKernelGGL((tiles_kernel<Op, DT, K, W, VEC, TR>),
                               dim3(unsigned(a.N * p.tiles_per_row)), block, 0, stream, a,
                               p.tiles_per_row);
            return;
        }
    }
    const int64_t groups = (a.N + p.rows_per_wg - 1) / p.rows_per_wg;
    hipLaunchKernelGGL((rows_kernel<Op, DT, K, W, VEC, TR, PAD>), dim3(unsigned(groups)), block,
                       p.lds_bytes, stream, a, p.rows_per_wg, p.wave_local);
}

template <class Op, typename DT, bool VEC, bool TR>
rlcs_status launch(const Args& a, const Plan& p, hipStream_t stream) {
    if constexpr (VEC && Op::kStaged == 0) {
        if (p.flat_R > 0) {
            const dim3 grid(unsigned((a.N + p.flat_R - 1) / p.flat_R));
            if constexpr (sizeof(DT) == 4) {
                if (p.flat_W == kLargeWaves) {
                    hipLaunchKernelGGL((flat_rows_kernel<Op, DT, Width<DT>::K, TR, kLargeWaves>), grid,
                                       dim3(kLargeWaves * kWave), 0, stream, a, p.flat_R, p.flat_magic);
                    return hipGetLastError() == hipSuccess ? RLCS_OK : RLCS_ERR_LAUNCH;
                }
            }
            hipLaunchKernelGGL((flat_rows_kernel<Op, DT, Width<DT>::K, TR, kSmallWaves>), grid,
                               dim3(kSmallWaves * kWave), 0, stream, a, p.flat_R, p.flat_magic);
            return hipGetLastError() == hipSuccess ? RLCS_OK : RLCS_ERR_LAUNCH;
        }
        if (p.wave_rows_log2T >= 0) {
            constexpr int64_t span = int64_t(kWave) * Width<DT>::K;
            const int64_t waves = (a.N * a.T + span - 1) / span;
            if constexpr (WaveRowsQuads<Op, DT, TR>::value) {
                if (a.N * a.T >= kWaveRowsQuadMinSteps && a.N * a.T <= kWaveRowsQuadSteps) {
                    hipLaunchKernelGGL((wave_rows_kernel<Op, DT, Width<DT>::K, TR, 4>),
                                       dim3(unsigned((waves + 3) / 4)), dim3(4 * kWave), 0, stream, a,
                                       p.wave_rows_log2T);
                    return hipGetLastError() == hipSuccess ? RLCS_OK : RLCS_ERR_LAUNCH;
                }
            }
            hipLaunchKernelGGL((wave_rows_kernel<Op, DT, Width<DT>::K, TR>), dim3(unsigned(waves)),
                               dim3(kWave), 0, stream, a, p.wave_rows_log2T);
            return hipGetLastError() == hipSuccess ? RLCS_OK : RLCS_ERR_LAUNCH;
        }
    }
    if constexpr (VEC && Op::kStaged == 0) {
        if (p.pad && !p.split) {
            if (p.waves == kSmallWaves) launch_w<Op, DT, true, TR, kSmallWaves, true>(a, p, stream);
            else launch_w<Op, DT, true, TR, kLargeWaves, true>(a, p, stream);
            return hipGetLastError() == hipSuccess ? RLCS_OK : RLCS_ERR_LAUNCH;
        }
    }
    if constexpr (Op::kStaged > 0 && Op::kSliced) {
        launch_w<Op, DT, VEC, TR, kStagedWaves>(a, p, stream);
    } else if constexpr (Op::kStaged > 0) {
        if (p.waves == kStagedWaves) launch_w<Op, DT, VEC, TR, kStagedWaves>(a, p, stream);
        else if (p.waves == kStagedMidWaves) launch_w<Op, DT, VEC, TR, kStagedMidWaves>(a, p, stream);
        else launch_w<Op, DT, VEC, TR, kSmallWaves>(a, p, stream);
    } else {
        if constexpr (OneWaveRows<Op>::value) {
            if (p.waves == 1) {
                launch_w<Op, DT, VEC, TR, 1>(a, p, stream);
                return hipGetLastError() == hipSuccess ? RLCS_OK : RLCS_ERR_LAUNCH;
            }
        }
        if (p.waves == kSmallWaves) launch_w<Op, DT, VEC, TR, kSmallWaves>(a, p, stream);
        else launch_w<Op, DT, VEC, TR, kLargeWaves>(a, p, stream);
    }
    return hipGetLastError() == hipSuccess ? RLCS_OK : RLCS_ERR_LAUNCH;
}

// LDS bytes of a staged policy's chunk with W waves: the larger of the two [steps, A] slices and
// the staged slots, which reuse the slices' bytes once they are reduced.
template <class Op, typename DT>
constexpr int64_t staged_lds_bytes(int W, int64_t A) {
    const int64_t E = int64_t(W) * kWave * Width<DT>::K;
    const int64_t per_block = 16 / int64_t(sizeof(DT));
    const int64_t cap = ((E + 1) * A + 3 * per_block) / per_block * per_block;  // see stage_chunk
    const int64_t slots = int64_t(sizeof(float)) * Op::kStaged * (E + 4);
    const int64_t slices = 2 * cap * int64_t(sizeof(DT));
    return slots > slices ? slots : slices;
}

// Sliced staging (long action axes), W waves: LDS elements of one array's slab of As actions
// (SlicedStager::cap), the widest slice (a multiple of 16 bytes of DT) whose two slabs fit in
// `budget` bytes, and the LDS bytes of a chunk (slabs or slots, which overlay them).
template <typename DT>
constexpr int64_t sliced_cap(int W, int64_t As) {
    const int64_t E = int64_t(W) * kWave * Width<DT>::K, per_block = 16 / int64_t(sizeof(DT));
    return ((E + 1) * As + per_block - 1) / per_block * per_block;
}
template <typename DT>
constexpr int64_t sliced_width(int W, int64_t budget) {
    // whole 128-byte lines of actions when one fits: a slice that ends inside a line leaves the
    // rest of that line to the next slice, which fetched it again from HBM (float32, A = 64 and
    // 256: 1.96 and 1.99 times the algorithmic bytes with 28-action slices)
    const int64_t per_line = 128 / int64_t(sizeof(DT));
    int64_t As = 0;
    while (2 * sliced_cap<DT>(W, As + per_line) * int64_t(sizeof(DT)) <= budget) As += per_line;
    if (As > 0) return As;
    const int64_t per_block = 16 / int64_t(sizeof(DT));
    As = per_block;
    while (2 * sliced_cap<DT>(W, As + per_block) * int64_t(sizeof(DT)) <= budget) As += per_block;
    return As;
}
template <class Op, typename DT>
constexpr int64_t sliced_lds_bytes(int W, int64_t As) {
    const int64_t E = int64_t(W) * kWave * Width<DT>::K;
    const int64_t slots = int64_t(sizeof(float)) * Op::kStaged * (E + 4);
    const int64_t slabs = 2 * sliced_cap<DT>(W, As) * int64_t(sizeof(DT));
    return slots > slabs ? slots : slabs;
}

template <class Op, typename DT>
rlcs_status dispatch_dt(Args& a, bool has_trunc, void* ws, size_t ws_bytes, hipStream_t stream) {
    constexpr int K = Width<DT>::K;
    constexpr int64_t E_small = int64_t(kSmallWaves) * kWave * K;
    constexpr int64_t E_large = int64_t(kLargeWaves) * kWave * K;
    const int64_t N = a.N, T = a.T;

    // Vector path: 16-byte data and output vectors, K-byte flag vectors.
    bool vec = true;
    for (int s = 0; s < Op::kSlots; ++s)
        if (Op::slot_used(s, has_trunc) && !aligned(a.in[s], 16)) vec = false;
    if (!aligned(a.out0, 16) || (a.out1 && !aligned(a.out1, 16))) vec = false;
    if (Op::kFlags && ((a.term && !aligned(a.term, K)) || (has_trunc && !aligned(a.trunc, K)))) vec = false;

    Plan p{};
    // Split rows: 4-wave tiles unless a row would have too many of them.
    const int64_t P_small = (T + E_small - 1) / E_small;
    const bool small_tiles = P_small <= kMaxSmallTilesPerRow;
    p.tiles_per_row = small_tiles ? P_small : (T + E_large - 1) / E_large;
    const bool slots_ok = N <= kWsSlots;  // one draw slot per row
    const size_t ws_need = slots_ok ? kWsRecordsOffset + size_t(N * p.tiles_per_row) * kWsRecordBytes
                                    : kWsRecordsOffset;
    const bool ws_ok = ws && ws_bytes >= ws_need && aligned(ws, 64);
    const int forced = g_variant;
    if constexpr (Op::kStaged > 0 && Op::kSliced) {
        // Long action axes: one-wave workgroups, the widest slice that fits the LDS budget.
        p.split = false;
        p.waves = kStagedWaves;
        a.A_slice = sliced_width<DT>(kStagedWaves, kSlicedLdsBudget);
        p.lds_bytes = size_t(sliced_lds_bytes<Op, DT>(kStagedWaves, a.A_slice));
    } else if constexpr (Op::kStaged > 0) {
        // Staged policies keep whole rows in one workgroup (chunk loop for long rows).
        p.split = false;
        if (staged_lds_bytes<Op, DT>(kSmallWaves, a.A) <= kStagedLdsBudget) p.waves = kSmallWaves;
        else if (staged_lds_bytes<Op, DT>(kStagedMidWaves, a.A) <= kStagedMidLdsBudget) p.waves = kStagedMidWaves;
        else if (staged_lds_bytes<Op, DT>(kStagedWaves, a.A) <= kStagedLdsBudget) p.waves = kStagedWaves;
        else return RLCS_ERR_INVALID_ARG;
        p.lds_bytes = size_t(staged_lds_bytes<Op, DT>(p.waves, a.A));
    } else {
        if (forced == 2) {
            if (!ws_ok) return RLCS_ERR_WORKSPACE;
            p.split = slots_ok;  // more rows than draw slots: whole rows
        } else if (forced == 1) {
            p.split = false;
        } else {
            p.split = ws_ok && slots_ok && T % K == 0 && T > E_large && N < kSplitBelowRows;
        }
        if (p.split) p.waves = small_tiles ? kSmallWaves : kLargeWaves;
        else if (T > E_small) p.waves = kLargeWaves;
        else if (OneWaveRows<Op>::value && T % K == 0 && (int64_t(kWave) * K) % T == 0 && T >= 32 * K)
            p.waves = 1;  // whole rows per wave, every chunk full
        else p.waves = kSmallWaves;
        p.lds_bytes = 0;
    }
    p.wave_rows_log2T = -1;
    p.flat_R = 0;
    p.flat_W = kSmallWaves;
    // Dense rows up to one sixteen-wave chunk (float32) or one wave (bfloat16), except powers of
    // two that tile a wave: the flat rows kernel. Measured against
    // the rows kernel (C harness, cold): GAE 4096x192 fp32 5.05 -> 4.62 us, 4096x252 5.97 -> 5.22,
    // 4096x500 10.04 -> 8.68, 4096x1000 16.59 -> 15.48, 4096x1024 16.13 -> 15.54; bf16 16384x200
    // 12.83 -> 11.14, 16384x504 24.98 -> 23.16; longer bf16 rows were within 2.5 % either way
    // (16384x1000 45.4 -> 44.2, 16384x2048 82.3 -> 83.4) and keep the rows kernel.
    // Rows whose length is not a multiple of K take it as well when a workgroup's rows can start
    // and end on vector boundaries (R a multiple of K / gcd(T, K), N*T a multiple of K).
    // float32 rows up to one sixteen-wave chunk (4096 steps) take it too, in sixteen-wave
    // ranges where four waves hold none, in place of one sixteen-wave rows-kernel workgroup per
    // row (same protocol, GAE): 4096x2000 36.2 -> 29.9 us, 2048x3000 32.7 -> 24.7, 1024x4096
    // 19.6 -> 17.1, 4096x1500 33.0 -> 24.7, 2048x2048 19.7 -> 17.0, 8192x1100 44.1 -> 34.0;
    // 64x4096 even (4.45 -> 4.43).
    const int64_t flat_max = sizeof(DT) == 4 ? E_large : int64_t(kWave) * K;
    if (Op::kStaged == 0 && !p.split && vec && T > K && T <= flat_max && (N * T) % K == 0 &&
        !((T & (T - 1)) == 0 && T <= int64_t(kWave) * K)) {
        int64_t gcd = K, b = T % K;
        while (b) { const int64_t r = gcd % b; gcd = b; b = r; }
        const int64_t step = K / gcd;  // rows per vector-aligned range
        int64_t R = E_small / T / step * step;
        int W = kSmallWaves;
        // float32 rows too long for `step` of them in four waves (more than 1024 steps, or more
        // than 256 that are not a multiple of K): sixteen waves hold 4096 steps
        if (R == 0 && sizeof(DT) == 4) {
            R = E_large / T / step * step;
            W = kLargeWaves;
        }
        const int64_t magic = ((int64_t(1) << flat_shift(W)) + T - 1) / T;
        if (R > 0 && (int64_t(W) * kWave * K - 1) * magic < (int64_t(1) << 32)) {
            p.flat_R = int(R);
            p.flat_W = W;
            p.flat_magic = uint32_t(magic);
            if ((N + R - 1) / R > INT32_MAX) return RLCS_ERR_INVALID_ARG;
        }
    }
    if (Op::kStaged == 0 && !p.split && vec && T >= K && T <= int64_t(kWave) * K && (T & (T - 1)) == 0) {
        // rows tile a wave exactly: the wave-rows kernel
        if ((N * T + int64_t(kWave) * K - 1) / (int64_t(kWave) * K) > INT32_MAX) return RLCS_ERR_INVALID_ARG;
        int l = 0;
        while ((int64_t(1) << l) < T) ++l;
        p.wave_rows_log2T = l;
    }
    if (p.split) {
        if (N * p.tiles_per_row > INT32_MAX) return RLCS_ERR_INVALID_ARG;
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
        // When a workgroup's rows do not fill its chunks exactly, every chunk still takes the
        // vector path lane by lane: only the lanes at the ragged ends of the workgroup's range
        // go element-wise.
        p.pad = vec && Op::kStaged == 0 && T >= K && (T % K != 0 || (p.rows_per_wg * T) % E != 0);
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

// Rows with a row stride (period) above T: the rows kernel over the positions n * period + t
// (the steps t >= T of each period are skipped), whole rows per workgroup; vector loads and
// stores where a lane's steps allow when the arrays are aligned, else element-wise.
template <class Op>
rlcs_status dispatch_strided_rows(Args& a, int64_t period, rlcs_dtype dtype, bool has_trunc,
                                  rlcs_stream_t stream) {
    if (a.N == 0 || a.T == 0) return RLCS_OK;
    if (period > kMaxT) return RLCS_ERR_INVALID_ARG;
    a.period = period;
    a.inv_period = 1.f / float(period);
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    auto run = [&](auto dt_tag) -> rlcs_status {
        using DT = decltype(dt_tag);
        constexpr int K = Width<DT>::K;
        Plan p{};
        p.split = false;
        const int64_t E_small = int64_t(kSmallWaves) * kWave * K;
        p.waves = (a.T <= E_small) ? kSmallWaves : kLargeWaves;
        const int64_t E = int64_t(p.waves) * kWave * K;
        const int64_t slack = (period % K == 0) ? 0 : K - 1;
        // as many rows as fit in one chunk: the last one's gap is not part of the range
        p.rows_per_wg = (a.T <= E - slack) ? (E - slack - a.T) / period + 1 : 1;
        if ((a.N + p.rows_per_wg - 1) / p.rows_per_wg > INT32_MAX) return RLCS_ERR_INVALID_ARG;
        p.wave_local = 0;
        p.lds_bytes = 0;
        p.wave_rows_log2T = -1;
        p.flat_R = 0;
        p.flat_W = kSmallWaves;
        // Vector path, lane by lane (lanes whose steps reach into a gap or past the range go
        // element-wise): T >= K, data and outputs 16-byte aligned, flags K-byte aligned.
        bool vec = a.T >= K;
        for (int i = 0; i < Op::kSlots; ++i)
            if (Op::slot_used(i, has_trunc) && !aligned(a.in[i], 16)) vec = false;
        if (!aligned(a.out0, 16) || (a.out1 && !aligned(a.out1, 16))) vec = false;
        if (Op::kFlags && ((a.term && !aligned(a.term, K)) || (has_trunc && !aligned(a.trunc, K)))) vec = false;
        p.pad = vec;
        auto go = [&](auto tr_tag) -> rlcs_status {
            constexpr bool TR = decltype(tr_tag)::value;
            return vec ? launch<Op, DT, true, TR>(a, p, s) : launch<Op, DT, false, TR>(a, p, s);
        };
        if constexpr (Op::kFlags) {
            if (has_trunc) return go(std::true_type{});
        }
        return go(std::false_type{});
    };
    if (dtype == RLCS_BF16) return run(bf16_t{});
    return run(float{});
}

inline Args make_args(int64_t N, int64_t T, float gamma, float lambda, float rho_bar, float c_bar) {
    Args a{};
    a.N = N;
    a.T = T;
    a.inv_T = T > 0 ? 1.f / float(T) : 0.f;
    a.period = T;
    a.inv_period = a.inv_T;
    a.p = Params{gamma, lambda, rho_bar, c_bar};
    return a;
}


}  // namespace host
}  // namespace rlcs
