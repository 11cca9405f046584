// Host side of the column scans (time-major layouts, vector eligibility traces): checks,
// the choice between whole columns per workgroup and split columns, and the launches.
#pragma once

#include <cmath>
#include <type_traits>

#include "rlcs_columns.h"
#include "rlcs_dispatch.h"

namespace rlcs {
namespace host {

// Column blocks (64 columns each) from which whole columns per workgroup already fill the GPU;
// below it, columns longer than one chunk are split into one-chunk tiles when a workspace is
// given. Never more than the workspace's per-block slots.
constexpr int64_t kColSerialBlocks = kWsSlots;
// Retrace from a quarter of that: its split tiles are eight waves of about 140 VGPRs, one
// workgroup per CU, while its whole-column walks run four-wave workgroups, two or more per CU.
// Time-major float32 T x N = 1024 x 32768 (512 blocks) 263 -> 195 us, 512 x 16384 (256 blocks)
// 60.7 -> 43.3 us. The other estimators gain or lose a few percent either way there.
constexpr int64_t kColSerialBlocksRetrace = kWsSlots / 4;

inline int64_t col_tiles(int64_t T) { return (T + kColL - 1) / kColL; }
inline int64_t col_split_tiles(int64_t T) { return (T + kColSplitL - 1) / kColSplitL; }

// Whole-column walks of at least this many chunks overlap each chunk's loads with the scan of
// the one before (shorter ones gain less than the unconditional continuation reads cost; four
// chunks gain 1-3%: vector traces 1 x 128 x 2^20 215 -> 208 us, time-major 128 x 32768).
constexpr int64_t kColPipeChunks = 4;

// Workspace bytes of a split column call: header and block slots, then two records per column
// per 32-step span (a bound on the split tiles, which are longer; 0 if the size does not fit in
// size_t).
inline size_t col_ws_need(int64_t J, int64_t T) {
    const int64_t P = col_tiles(T);
    if (J <= 0 || P <= 0) return kWsRecordsOffset;
    if (P > INT64_MAX / J || P * J > int64_t(SIZE_MAX / kWsRecordBytes) / 2) return 0;
    return kWsRecordsOffset + size_t(P * J) * kWsRecordBytes;
}

// Narrow column groups (whole columns, no workspace) when the columns fit in one 16-wave chunk
// (256 steps) and the groups give one or two workgroups per CU. Columns of at most 64 (128)
// steps take 4-wave (8-wave) workgroups: 16 waves would leave half or more of them idle
// (128 x 8192: 8.0 us with 16 waves, 6.6 with 8). Longer columns walk chunk
// after chunk, one workgroup per CU, and the split tiles are faster there; with more groups
// the 1024-thread workgroups queue behind each other. C harness, cold, time-major GAE, narrow
// against split: 256 x 4096 6.84 us against 8.23; 128 x 8192 8.04 against 8.06; 256 x 16384
// 19.6 against 17.7; 512 x 4096 15.0 against 11.5; 2048 x 4096 55.4 against 41.7.
constexpr int64_t kNarrowMinGroups = 256;
constexpr int64_t kNarrowMaxGroups = 512;
// Split calls whose 64-column tiles give fewer workgroups than this (one per CU) split narrow
// groups instead, with four (two) times the workgroups: T x N = 4096 x 64 float32 takes 6.2 us
// instead of 7.4, 2048 x 128 6.4 instead of 7.3; at 256 workgroups and more (1024 x 1024,
// 4096 x 256, 8192 x 128, 32768 x 64) the 64-column tiles are 10-25% faster. So do calls of
// fewer than 64 columns, whose one 64-column block leaves lanes idle: 16384 x 32 7.4 us instead
// of 10.1.
constexpr int64_t kNarrowSplitBelowWgs = 256;
// Narrow walks of at least this many chunks overlap each chunk's loads with the scan before.
constexpr int64_t kNarrowPipeChunks = 4;

template <typename DT>
inline int64_t narrow_groups(int64_t J) { return (J + narrow_cols<DT>() - 1) / narrow_cols<DT>(); }

// Steps of a 16-wave narrow chunk (the same for both dtypes).
constexpr int64_t kNarrowChunk = int64_t(kWave / narrow_cols<float>()) * 16 * (narrow_cols<float>() / 4);
static_assert(kNarrowChunk == int64_t(kWave / narrow_cols<bf16_t>()) * 16 * (narrow_cols<bf16_t>() / 4),
              "narrow chunks hold the same number of steps in both dtypes");

template <class Op, typename DT, bool TR, bool NT>
void narrow_launch_nt(const Args& a, const ColGeom& g, hipStream_t s) {
    constexpr int C = narrow_cols<DT>();
    constexpr int K = C / 4;  // 4 float32 or 8 bfloat16 steps per lane: 16 steps per wave
    constexpr int G = kWave / C;
    const dim3 grid(unsigned(narrow_groups<DT>(g.J)));
    if (a.T <= int64_t(G) * 4 * K) {  // one 4-wave chunk
        hipLaunchKernelGGL((cols_narrow_kernel<Op, DT, K, 4, TR, false, NT>), grid, dim3(4 * kWave), 0,
                           s, a, g, int64_t(grid.x));
        return;
    }
    if (a.T <= int64_t(G) * 8 * K) {  // one 8-wave chunk
        hipLaunchKernelGGL((cols_narrow_kernel<Op, DT, K, 8, TR, false, NT>), grid, dim3(8 * kWave), 0,
                           s, a, g, int64_t(grid.x));
        return;
    }
    const int64_t chunks = (a.T + int64_t(G) * 16 * K - 1) / (int64_t(G) * 16 * K);
    if (chunks >= kNarrowPipeChunks) {
        hipLaunchKernelGGL((cols_narrow_kernel<Op, DT, K, 16, TR, true, NT>), grid, dim3(16 * kWave), 0,
                           s, a, g, int64_t(grid.x));
    } else {
        hipLaunchKernelGGL((cols_narrow_kernel<Op, DT, K, 16, TR, false, NT>), grid, dim3(16 * kWave), 0,
                           s, a, g, int64_t(grid.x));
    }
}

// Split tiles publish block aggregates for long look-backs when a look-back may pass more than
// this many tiles before the product of their betas underflows to 0.
constexpr int64_t kColLiftTiles = 32;

// Whether a look-back over P tiles of kColSplitL steps can be long: each step's beta is at most
// gamma * lambda * max(1, c_bar) for every column scan, and a product of betas below about
// 1.4e-45 is 0 in float32.
inline bool col_lift(const Params& p, int64_t P) {
    if (P <= kColLiftTiles) return false;
    const double bmax = double(p.gamma) * double(p.lambda) * (p.c_bar > 1.f ? double(p.c_bar) : 1.0);
    if (!(bmax < 1.0)) return true;
    if (bmax <= 0.0) return false;
    const double tiles = 104.0 / (double(kColSplitL) * -std::log(bmax)) + 1.0;
    return tiles > double(kColLiftTiles);
}

template <class Op, typename DT, bool TR, bool NT>
void col_launch_nt(const Args& a, const ColGeom& g, bool split, int64_t blocks, hipStream_t s) {
    const dim3 block(kColW * kWave);
    if (split) {
        const int64_t P = col_split_tiles(a.T);
        const dim3 grid(unsigned(blocks * P)), tile_block(kColSplitW * kWave);
        if (col_lift(a.p, P))
            hipLaunchKernelGGL((cols_tiles_kernel<Op, DT, kColK, kColSplitW, TR, true, NT>), grid,
                               tile_block, 0, s, a, g, blocks);
        else
            hipLaunchKernelGGL((cols_tiles_kernel<Op, DT, kColK, kColSplitW, TR, false, NT>), grid,
                               tile_block, 0, s, a, g, blocks);
    } else if (col_tiles(a.T) >= kColPipeChunks) {
        hipLaunchKernelGGL((cols_rows_kernel<Op, DT, kColK, kColW, TR, true, NT>), dim3(unsigned(blocks)),
                           block, 0, s, a, g);
    } else {
        hipLaunchKernelGGL((cols_rows_kernel<Op, DT, kColK, kColW, TR, false, NT>), dim3(unsigned(blocks)),
                           block, 0, s, a, g);
    }
}

// Split tiles over narrow column groups, a block being one narrow group: TL-step tiles of
// TL / 16 waves (4 lane groups x 4 float32 steps, or 2 x 8 bfloat16 steps, per wave).
template <class Op, typename DT, bool TR, bool NT, int TL>
void narrow_split_launch_tl(const Args& a, const ColGeom& g, int64_t nblocks, hipStream_t s) {
    constexpr int C = narrow_cols<DT>();
    constexpr int K = C / 4;
    constexpr int G = kWave / C;
    constexpr int W = TL / (G * K);
    static_assert(G * W * K == TL, "a narrow split tile is a whole number of waves");
    const int64_t P = (a.T + TL - 1) / TL;
    const dim3 grid(unsigned(nblocks * P)), block(W * kWave);
    // Tiles dealt statically to XCDs, or drawn in arrival order (always under variant 4). Both
    // orders measured, time-major float32 GAE, C harness, cold, drawn against dealt (T x N):
    // 128-step tiles 4096 x 128 7.99 us against 6.72, 8192 x 64 7.23 against 6.95; 64-step
    // tiles in at most 16 tiles per column 1024 x 64 5.58 against 5.09, 1024 x 40 5.63 against
    // 5.00; 64-step tiles in more: 4096 x 64 6.25 against 6.69, 2048 x 128 6.34 against 6.62,
    // 4096 x 32 6.20 against 6.47, 8192 x 32 6.87 against 6.98. Dealt, 4096 x 64 fetches 0.99
    // times its algorithmic bytes, drawn 1.59 times, and still runs faster.
    auto dealt = [&](auto kernel) {
        return int(g_variant == 0 && P % 8 == 0 && (TL > kColSplitL || P <= 16) &&
                   nblocks * P <= resident_groups(kernel, W * kWave));
    };
    if (col_lift(a.p, P)) {
        const auto kernel = cols_narrow_tiles_kernel<Op, DT, K, W, TR, true, NT>;
        hipLaunchKernelGGL(kernel, grid, block, 0, s, a, g, nblocks, dealt(kernel));
    } else {
        const auto kernel = cols_narrow_tiles_kernel<Op, DT, K, W, TR, false, NT>;
        hipLaunchKernelGGL(kernel, grid, block, 0, s, a, g, nblocks, dealt(kernel));
    }
}

// Narrow split grids of more than this many 64-step tiles take 128-step tiles (half the
// workgroups, half the look-back chain): T x N = 8192 x 64 float32 7.3 us instead of 8.2, and
// 9.9 instead of 11.4 without flags and gamma = lambda = 1; at 256 tiles and fewer the 64-step
// tiles are 3-6% faster on flagged data (4096 x 64, 2048 x 128).
constexpr int64_t kNarrowSplitLongAbove = 256;

template <class Op, typename DT, bool TR, bool NT>
void narrow_split_launch_nt(const Args& a, const ColGeom& g, int64_t nblocks, hipStream_t s) {
    if (nblocks * col_split_tiles(a.T) > kNarrowSplitLongAbove)
        return narrow_split_launch_tl<Op, DT, TR, NT, 2 * kColSplitL>(a, g, nblocks, s);
    narrow_split_launch_tl<Op, DT, TR, NT, kColSplitL>(a, g, nblocks, s);
}

// Plain-store kernels exist only for the eligibility-trace policy, the one that vector traces
// (whose rows may hold fewer than 32 features) run on.
template <class Op>
constexpr bool kPlainStores = std::is_same<Op, ForwardOp<true, false>>::value;

template <class Op, typename DT, bool TR>
void narrow_launch(const Args& a, const ColGeom& g, hipStream_t s) {
    if constexpr (kPlainStores<Op>) {
        if (!g.nt_store) return narrow_launch_nt<Op, DT, TR, false>(a, g, s);
    }
    narrow_launch_nt<Op, DT, TR, true>(a, g, s);
}

template <class Op, typename DT, bool TR>
void narrow_split_launch(const Args& a, const ColGeom& g, int64_t nblocks, hipStream_t s) {
    if constexpr (kPlainStores<Op>) {
        if (!g.nt_store) return narrow_split_launch_nt<Op, DT, TR, false>(a, g, nblocks, s);
    }
    narrow_split_launch_nt<Op, DT, TR, true>(a, g, nblocks, s);
}

template <class Op, typename DT, bool TR>
void col_launch(const Args& a, const ColGeom& g, bool split, int64_t blocks, hipStream_t s) {
    if constexpr (kPlainStores<Op>) {
        if (!g.nt_store) return col_launch_nt<Op, DT, TR, false>(a, g, split, blocks, s);
    }
    col_launch_nt<Op, DT, TR, true>(a, g, split, blocks, s);
}

template <class Op>
rlcs_status col_dispatch(Args& a, const ColGeom& g, rlcs_dtype dtype, bool has_trunc, void* ws,
                         size_t ws_bytes, rlcs_stream_t stream) {
    if (g.J == 0 || a.T == 0) return RLCS_OK;
    const int64_t blocks = (g.J + kWave - 1) / kWave;
    const int64_t P = col_tiles(a.T);
    const size_t need = col_ws_need(g.J, a.T);
    const bool ws_ok = ws && need > 0 && ws_bytes >= need && aligned(ws, 64) &&
                       blocks <= int64_t(UINT32_MAX) / P;
    const int forced = g_variant;
    const int64_t ngroups = dtype == RLCS_BF16 ? narrow_groups<bf16_t>(g.J) : narrow_groups<float>(g.J);
    if (forced == 3 || (forced == 0 && a.T <= kNarrowChunk && ngroups >= kNarrowMinGroups &&
                        ngroups <= kNarrowMaxGroups)) {
        if (ngroups > INT32_MAX) return RLCS_ERR_INVALID_ARG;
        hipStream_t s = reinterpret_cast<hipStream_t>(stream);
        const bool tr = Op::kFlags && has_trunc;
        if (dtype == RLCS_BF16) {
            if (tr) narrow_launch<Op, bf16_t, true>(a, g, s);
            else narrow_launch<Op, bf16_t, false>(a, g, s);
        } else {
            if (tr) narrow_launch<Op, float, true>(a, g, s);
            else narrow_launch<Op, float, false>(a, g, s);
        }
        return hipGetLastError() == hipSuccess ? RLCS_OK : RLCS_ERR_LAUNCH;
    }
    bool split;
    if (forced == 2) {
        if (!ws_ok) return RLCS_ERR_WORKSPACE;
        split = blocks <= kWsSlots;  // more blocks than slots: whole columns
    } else if (forced == 1) {
        split = false;
    } else {
        const int64_t serial = std::is_same_v<Op, RetraceOp> ? kColSerialBlocksRetrace : kColSerialBlocks;
        split = P > 1 && ws_ok && blocks < serial;
    }
    if (split && col_split_tiles(a.T) == 1) split = false;  // one tile: a whole-column walk
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    const bool tr = Op::kFlags && has_trunc;
    // Fewer split tiles than CUs, or one partly filled 64-column block: split the narrow groups
    // instead. Forced by variant 4 whenever the workspace allows.
    const bool nsplit_ok = ws_ok && ngroups <= kWsSlots && col_split_tiles(a.T) > 1;
    const bool nsplit_auto =
        split && (blocks * col_split_tiles(a.T) < kNarrowSplitBelowWgs || g.J < kWave);
    if (forced == 4 && !ws_ok) return RLCS_ERR_WORKSPACE;
    if (nsplit_ok && (forced == 4 || (forced == 0 && nsplit_auto))) {
        if (ngroups * col_split_tiles(a.T) > INT32_MAX) return RLCS_ERR_INVALID_ARG;
        a.ws = ws;
        if (dtype == RLCS_BF16) {
            if (tr) narrow_split_launch<Op, bf16_t, true>(a, g, ngroups, s);
            else narrow_split_launch<Op, bf16_t, false>(a, g, ngroups, s);
        } else {
            if (tr) narrow_split_launch<Op, float, true>(a, g, ngroups, s);
            else narrow_split_launch<Op, float, false>(a, g, ngroups, s);
        }
        return hipGetLastError() == hipSuccess ? RLCS_OK : RLCS_ERR_LAUNCH;
    }
    if (split) {
        if (blocks * P > INT32_MAX) return RLCS_ERR_INVALID_ARG;
        a.ws = ws;
    } else if (blocks > INT32_MAX) {
        return RLCS_ERR_INVALID_ARG;
    }
    if (dtype == RLCS_BF16) {
        if (tr) col_launch<Op, bf16_t, true>(a, g, split, blocks, s);
        else col_launch<Op, bf16_t, false>(a, g, split, blocks, s);
    } else {
        if (tr) col_launch<Op, float, true>(a, g, split, blocks, s);
        else col_launch<Op, float, false>(a, g, split, blocks, s);
    }
    return hipGetLastError() == hipSuccess ? RLCS_OK : RLCS_ERR_LAUNCH;
}

// Strided [N, T] geometry: element (n, t) of every [N, T] array of the call (data, flags,
// continuation values, outputs) at n * stride_n + t * stride_t, both strides >= 1 and one
// dimension nested in the other (stride_n >= T * stride_t, or stride_t >= N * stride_n), so
// that distinct (n, t) are distinct elements. Column n is environment n (one column per batch
// row), its flags laid out like its data. `dense`: the plain row-major layout.
inline rlcs_status check_strided(int64_t N, int64_t T, int64_t sn, int64_t st, rlcs_dtype dtype,
                                 std::initializer_list<const void*> data,
                                 std::initializer_list<const void*> outs, ColGeom& g, bool& dense) {
    if (N < 0 || T < 0) return RLCS_ERR_INVALID_ARG;
    if (dtype != RLCS_F32 && dtype != RLCS_BF16) return RLCS_ERR_DTYPE;
    if (sn < 1 || st < 1 || T > kMaxT) return RLCS_ERR_INVALID_ARG;
    if (N > 0 && T > 0) {
        if ((N - 1) > INT64_MAX / sn || (T - 1) > INT64_MAX / st) return RLCS_ERR_INVALID_ARG;
        const int64_t en = (N - 1) * sn, et = (T - 1) * st;
        if (en > INT64_MAX - et) return RLCS_ERR_INVALID_ARG;
        const bool rows_outer = T <= sn / st;   // sn >= T * st
        const bool steps_outer = N <= st / sn;  // st >= N * sn
        if (!rows_outer && !steps_outer) return RLCS_ERR_INVALID_ARG;
    }
    const size_t es = dtype_size(dtype);
    for (const void* p : data)
        if (p && !aligned(p, es)) return RLCS_ERR_INVALID_ARG;
    for (const void* p : outs)
        if (p && !aligned(p, 4)) return RLCS_ERR_INVALID_ARG;
    g = ColGeom{N, 1, st, sn, 0, 0, 1, 1};
    dense = st == 1 && sn == T;
    return RLCS_OK;
}

}  // namespace host
}  // namespace rlcs
