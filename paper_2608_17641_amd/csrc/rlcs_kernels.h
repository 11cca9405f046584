// The two kernel shapes that run every estimator.
//
// Both treat the [N, T] buffer as one flat array of N*T steps and run a segmented scan over it:
// each lane owns K consecutive steps (one 16-byte vector per input), a wave owns 64*K steps and
// a workgroup of W waves a chunk of E = W*64*K steps. Per chunk:
//   1. load every input once (coalesced vector loads), with the carry-source neighbour of the
//      lane's edge step taken from the adjacent lane by shuffle, or from memory at a wave edge;
//   2. build alpha, beta in registers (the policy's `build`);
//   3. compose the lane's K steps serially into one affine map;
//   4. scan those maps across the wave with shuffles (6 steps);
//   5. compose the waves' maps through LDS;
//   6. apply the carry entering the chunk and run the recurrence serially inside each lane;
//   7. the policy's epilogue and one vector store per output.
//
// rows kernel  : each workgroup owns whole rows and walks them chunk by chunk from the carry
//                source, passing the carry between chunks in LDS. Needs no workspace. Rows
//                may also lie a stride (`period`) apart; with PAD, chunks that the rows do not
//                fill exactly still run vector loads, each lane deciding for itself (Chunk).
// tiles kernel : rows split into tiles of one chunk each (the last tile of a row may be
//                shorter), one workgroup per tile. A tile whose carry-source edge is not the
//                row's edge needs the carry from the tiles after it (backward) or before it
//                (forward) in the same row: every tile publishes its composed map to the
//                workspace as soon as step 5 is done, and a waiting tile composes its
//                neighbours' maps, nearest first, until it meets a map with beta = 0 (an episode
//                or row edge). Only maps are exchanged, never partial results, so the
//                association order is fixed and results are reproducible bit for bit. Tile
//                order within a row comes from the row's atomic ticket, so a tile only ever
//                waits for tiles that started before it.
#pragma once

#include <type_traits>

#include "rlcs_estimators.h"

namespace rlcs {

// Workspace layout (zero-filled once by the caller), shared by the split kernels of every
// entry point so that one workspace serves calls of any kind and shape:
//   header (64 bytes): a reserved word and an error flag;
//   kWsSlots draw slots of 64 bytes, one per row (row tiles) or per 64-column block (column
//   tiles), each holding one 64-bit draw word: generation << 32 | tickets drawn in this call;
//   from kWsRecordsOffset, the records: two 64-bit words per tile, (tag0 << 32 | bits(a)) and
//   (tag1 << 32 | bits(b)), at index x * n + i for row (column) i of the call's n, with x the
//   tile (rows) or the tile or block aggregate (columns, rlcs_columns.h).
// A workgroup draws its ticket and its slot's generation with one relaxed atomic add; the last
// drawer of a slot stores (gen + 1, 0), so the next call on the same stream finds the slot
// ready with a new generation, and no workgroup counts anything at its end. The slots a call
// does not draw from are moved on to gen + 1 as well (advance_idle_slots), so every slot always
// holds the same generation: the number of split calls made on the workspace, which names one
// call of its whole history (modulo 2^30). A record word is valid for the current call when its
// tag is the call's: tag0 = 2*gen + 1 (row tiles; 2*gen + 2 for column tiles) on the word of
// a, tag1 = tag0 + n * kTagMix on the word of b. Each word is checked on its own, so each tag
// must name the call by itself: a reader may load one word before the writer's store and the
// other after it, and a stale word whose tag matched the current call's would then pair with a
// current one. With per-slot generations that could happen (a word of another call, of another
// n, written when its slot stood at the generation the reader's slot stands at now); with the
// generation shared by all slots, no earlier call wrote a word with either current tag.
struct WsHeader {
    uint64_t reserved;
    uint32_t error;  // set to 1 if a call found the workspace in an inconsistent state
    uint32_t pad[13];
};
static_assert(sizeof(WsHeader) == 64, "workspace header is 64 bytes");
constexpr size_t kWsRecordBytes = 16;
constexpr int64_t kWsSlots = 1024;  // rows or column blocks a split call may have
constexpr size_t kWsSlotsBytes = size_t(kWsSlots) * 64;
constexpr size_t kWsRecordsOffset = sizeof(WsHeader) + kWsSlotsBytes;
constexpr uint32_t kGenMask = 0x3fffffffu;
constexpr uint32_t kTagMix = 0x9e3779b1u;  // odd: distinct n give distinct tag1

template <typename T>
__device__ __forceinline__ T ld_relaxed(const T* p) {
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
template <typename T>
__device__ __forceinline__ void st_relaxed(T* p, T v) {
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Ticket of a workgroup among the n_tiles workgroups of a call that draw from `word`, and the
// slot's generation for this call; one relaxed atomic, by one thread.
__device__ __forceinline__ uint32_t draw_ticket(uint64_t* word, int64_t n_tiles, uint32_t& gen) {
    const uint64_t old = __hip_atomic_fetch_add(word, uint64_t(1), __ATOMIC_RELAXED,
                                                __HIP_MEMORY_SCOPE_AGENT);
    const uint32_t ticket = uint32_t(old);
    gen = uint32_t(old >> 32) & kGenMask;
    if (ticket == uint32_t(n_tiles - 1)) st_relaxed(word, uint64_t((gen + 1u) & kGenMask) << 32);
    return ticket;
}

// Marks, in the workspace header's error word, a full-form Retrace call that met an action
// outside [0, A) (value 2; the call takes that step's Q and pi as 0).
__device__ __forceinline__ void report_bad_action(void* ws) {
    st_relaxed(&reinterpret_cast<WsHeader*>(ws)->error, 2u);
}

__device__ __forceinline__ uint64_t* draw_word(void* ws, int64_t slot) {
    return reinterpret_cast<uint64_t*>(reinterpret_cast<char*>(ws) + sizeof(WsHeader) + slot * 64);
}

// Moves the slots from `used` on, which no workgroup of this call draws from, to generation
// gen + 1, the generation the last drawer of each used slot leaves behind: run by every lane of
// one wave per workgroup, once the workgroup's own draw has returned `gen` (all slots stand at
// the same generation). The slots are spread over the grid, a few stores per workgroup.
__device__ __forceinline__ void advance_idle_slots(void* ws, int64_t used, uint32_t gen, int lane) {
    const uint64_t next = uint64_t((gen + 1u) & kGenMask) << 32;
    for (int64_t s = used + int64_t(blockIdx.x) * kWave + lane; s < kWsSlots;
         s += int64_t(gridDim.x) * kWave)
        st_relaxed(draw_word(ws, s), next);
}

// Lane l of a wave owns the l-th group of K steps of the wave's span for forward scans and the
// (63-l)-th for backward scans, so that in both directions the carry flows from lane l-1 to
// lane l and the wave scan is a prefix scan over lanes.
template <bool kBack>
__device__ __forceinline__ int lane_group(int lane) { return kBack ? (kWave - 1 - lane) : lane; }

// A hook that does nothing.
struct Nop {
    __device__ void operator()() const {}
};

// Row and step of flat positions relative to a base position whose row and step are known:
// position base.pos + d (0 <= d, base.t + d < 2^31) is in row base.row + q at step r, where
// (q, r) = divmod(base.t + d, T). The quotient comes from an fp32 reciprocal (inv_T = 1/T) and
// is corrected by at most one in either direction, which makes it exact for the offsets that
// occur here (base.t + d < T + 16*64*K, or < 2^31 with a quotient below 2).
struct RowBase {
    int64_t pos, row, t;
};

__device__ __forceinline__ void row_and_step(const RowBase& b, int64_t p, int64_t T, float inv_T,
                                             int64_t& row, int64_t& t) {
    const uint32_t u = uint32_t(b.t + (p - b.pos));
    const uint32_t Tu = uint32_t(T);
    uint32_t q = uint32_t(float(u) * inv_T);
    int64_t r = int64_t(u) - int64_t(q) * int64_t(Tu);
    if (r < 0) { --q; r += Tu; }
    else if (r >= int64_t(Tu)) { ++q; r -= Tu; }
    row = b.row + q;
    t = r;
}

// Per-thread state of one chunk between the local scan and the carry application.
//
// FULL chunks (every step of the chunk in range, 16-byte aligned data, T >= K) take a
// branch-free path: one vector load per input, issued back to back, and at most one row edge
// per lane, whose per-row value is loaded unconditionally from a clamped row index. Other
// chunks (the ragged ends of a range) take the masked element-wise path.
// PAD: every chunk takes the vector path, lane by lane. Rows lie `a.period` steps apart
// (period >= T; the steps t >= T of a period are a gap). A lane whose K steps are all in the
// workgroup's range [lo, hi) and, with gaps, all among the first T steps of one row takes the
// vector path; so does, without gaps, a lane at a ragged end of the range whose vector lies
// inside the array (its steps outside the range are masked off: the identity map, no stores).
// Any other lane (a vector that reaches into a gap or past the array, or one wholly outside
// the range) takes the element-wise path for its steps in range, which may be none.
template <class Op, typename DT, int K, int W, bool VEC, bool TR, bool PAD = false>
struct Chunk {
    static_assert(!PAD || (VEC && Op::kStaged == 0), "padded rows: vector path, unstaged policies");
    static constexpr bool kBack = Op::kBackward;
    static constexpr int NS = Op::kSlots;
    static constexpr int NB = Op::kNbr > 0 ? Op::kNbr : 1;
    static constexpr uint32_t kAll = (K == 32) ? 0xffffffffu : ((1u << K) - 1u);
    static constexpr int kStride = W * kWave * K + 4;  // staged slot stride (floats)

    float d[NS][K];
    float B[K];
    float nb[NB];
    float al[K], be[K];
    uint32_t term, trunc, edge, valid;
    int64_t p0;
    int sidx;            // p0 - chunk_lo: the lane's first step within the chunk
    const float* stage;  // staged slots (policies with kStaged > 0)
    // Eight outputs per lane, unstaged policies: a wave of a full chunk whose lanes all store
    // whole vectors holds 512 consecutive outputs, stored as whole lines through its LDS slot.
    static constexpr bool kLineStores = K == 8 && Op::kStaged == 0;
    f32x4* oslot = nullptr;
    Pair incl;     // lanes 0..lane of this wave composed (lane 0 innermost)
    Pair wave_in;  // waves between this wave and the chunk's carry-source edge

    // Forward policies with a neighbour (the done flag of the step before), full chunks of
    // several waves: lane 0 of a wave after the first does not read that flag from memory (a
    // 128-byte line that the wave before streams past L2 as well). It builds its first step
    // as if no flag cut it, every wave stores its last step's done flag in LDS with its map,
    // and after the barrier a wave whose predecessor's last step is done scales the beta of
    // its first step, of every lane's inclusive map and of its wave map by 0: the innermost
    // beta only ever multiplies the beta part of a composition, so this equals building
    // with it (bit for bit). `defer_chunk_`: the chunk defers; `defer_`: this wave does.
    // Four-wave chunks only: with sixteen waves it made one-row-per-workgroup calls slower
    // (eligibility traces 1024 x 4096 fp32 9.9 -> 12.8 us, 256 x 8192 6.6 -> 7.2), unexplained.
    static constexpr bool kCanDefer = !kBack && Op::kNbr > 0 && Op::kStaged == 0 && !PAD && W == 4;
    bool defer_chunk_ = false, defer_ = false;

    // Whether lane 0 must read the carry-source neighbour of its edge step from memory: only
    // if that step is in range and not a row edge (then the neighbour is in the same row,
    // hence inside the array), and the wave does not take it from LDS later.
    __device__ bool needs_nbr(int lane) const {
        const int ke = kBack ? K - 1 : 0;
        return Op::kNbr > 0 && Op::kStaged == 0 && lane == 0 && bit(valid, ke) && !bit(edge, ke) &&
               !(kCanDefer && defer_);
    }

    // Staged slot s (Op::staged_index(s) >= 0) of the lane's K steps, from LDS.
    __device__ void read_staged(int s, uint32_t mask, bool full) {
        const float* src = stage + Op::staged_index(s) * kStride + sidx;
#pragma unroll
        for (int k = 0; k < K; ++k) d[s][k] = (full || bit(mask, k)) ? src[k] : 0.f;
    }

    // Raw words of a FULL chunk's loads, between load_full and convert_full.
    static constexpr int kWords = K * int(sizeof(DT)) / 4;
    static constexpr int kTS = TR ? Op::kTruncSlot : -1;
    uint32_t w_[NS][kWords];
    uint32_t tw_[(K + 3) / 4], rw_[(K + 3) / 4];
    float rv_raw_;
    int ke_;

    // Step 1 for a chunk whose steps are all in range. The flag and data loads go out first
    // (their addresses need nothing but p0); the row bookkeeping, the per-row value and the
    // neighbour load follow while they are in flight; a lane reads its truncation
    // continuations only if one of its steps is truncated. No loaded value is used before every
    // load of the lane has been issued. Staged policies convert later (convert_full after the
    // stage is complete), so that nothing waits for a load while the staging copies, issued
    // after the flags, are in flight; they read the continuations unconditionally, since
    // choosing by the flags would wait for the copies.
    template <class BaseFn, class PreFn>
    __device__ void load_full(const Args& a, int64_t lo, int64_t hi, BaseFn&& base_of, int lane,
                              float (&nraw)[Op::kNbrRaw], PreFn&& pre) {
        const int64_t T = a.T;
        int64_t row = 0, t = 0;
        uint32_t in_range = kAll;
        bool deferred = false;  // row and step found once the loads are out
        if constexpr (PAD) {
            bool vector = false, skip = false;
            if (p0 >= lo && p0 + K <= hi) {
                if (a.period == T) {
                    vector = deferred = true;  // no gaps: a lane in range takes the vector path
                } else {
                    row_and_step(base_of(), p0, a.period, a.inv_period, row, t);
                    if (t + K <= T) vector = true;
                    else skip = t >= T && t + K <= a.period;  // wholly in a gap
                }
            } else if (p0 + K <= lo || p0 >= hi) {
                skip = true;  // wholly outside the range
            } else if (a.period == T && p0 >= 0 && p0 + K <= a.N * T) {
                // a ragged end of a range without gaps, inside the array
                vector = true;
                if (p0 < lo) {
                    in_range &= (kAll << uint32_t(lo - p0)) & kAll;
                    const RowBase b = base_of();  // the row before the range's first one
                    row_and_step(RowBase{b.pos - T, b.row - 1, b.t}, p0, T, a.inv_T, row, t);
                } else {
                    row_and_step(base_of(), p0, T, a.inv_T, row, t);
                }
                if (p0 + K > hi) in_range &= kAll >> uint32_t(p0 + K - hi);
            }
            if (skip) {  // no step to do: no loads, the identity map, no stores
                valid = 0;
                edge = 0;
                ke_ = -1;
                rv_raw_ = 0.f;
                trunc = 0;
#pragma unroll
                for (int i = 0; i < (K + 3) / 4; ++i) { tw_[i] = 0u; rw_[i] = 0u; }
#pragma unroll
                for (int s = 0; s < NS; ++s)
#pragma unroll
                    for (int i = 0; i < kWords; ++i) w_[s][i] = 0u;
                convert_full(a);
                return;
            }
            if (!vector) {
                load_masked(a, lo, hi, base_of, lane, nraw, pre);
                return;
            }
        }
        valid = in_range;
        // A missing optional array is read from in[0] instead (in bounds) and the value dropped.
        const uint8_t* fallback = reinterpret_cast<const uint8_t*>(a.in[0]);
        if (Op::kFlags && TR) load_flag_words<K>(a.trunc, p0, rw_);
        if (Op::kFlags) load_flag_words<K>(a.term ? a.term : fallback, p0, tw_);
        pre();
#pragma unroll
        for (int s = 0; s < NS; ++s)
            if (Op::slot_used(s, TR) && s != kTS) load_words<DT, K>(a.in[s], p0, w_[s]);

        // at most one row edge among the K steps (T >= K)
        if constexpr (!PAD) row_and_step(base_of(), p0, T, a.inv_T, row, t);
        else if (deferred) row_and_step(base_of(), p0, T, a.inv_T, row, t);
        ke_ = -1;
        int64_t row_e = row;
        if (kBack) {
            if (t + K - 1 >= T - 1) ke_ = int(T - 1 - t);
        } else {
            if (t == 0) ke_ = 0;
            else if (t + K - 1 >= T) { ke_ = int(T - t); row_e = row + 1; }
        }
        edge = ke_ >= 0 ? (1u << ke_) : 0u;
        const bool has_rv = Op::kRowValue && a.row_value;
        rv_raw_ = load_one<DT>(has_rv ? a.row_value : a.in[0], min(row_e, a.N - 1));
        if (needs_nbr(lane)) Op::template nbr_load_raw<DT>(a, kBack ? p0 + K : p0 - 1, nraw);
        if constexpr (Op::kStaged > 0) {
            if constexpr (kTS >= 0) load_words<DT, K>(a.in[kTS], p0, w_[kTS]);
        } else {
            trunc = (Op::kFlags && TR) ? flag_mask<K>(rw_) : 0u;
            if constexpr (kTS >= 0) {
                if (trunc) load_words<DT, K>(a.in[kTS], p0, w_[kTS]);
                else {
#pragma unroll
                    for (int i = 0; i < kWords; ++i) w_[kTS][i] = 0u;
                }
            }
            convert_full(a);
        }
    }

    // The conversions of load_full.
    __device__ void convert_full(const Args& a) {
        if constexpr (Op::kStaged > 0) trunc = (Op::kFlags && TR) ? flag_mask<K>(rw_) : 0u;
#pragma unroll
        for (int s = 0; s < NS; ++s) {
            if (Op::staged_index(s) >= 0) continue;  // read from LDS in the scan
            if (Op::slot_used(s, TR)) unpack_words<DT, K>(w_[s], d[s]);
            else {
#pragma unroll
                for (int k = 0; k < K; ++k) d[s][k] = 0.f;
            }
        }
        term = (Op::kFlags && a.term) ? flag_mask<K>(tw_) : 0u;
        const float rv = (Op::kRowValue && a.row_value) ? rv_raw_ : 0.f;
#pragma unroll
        for (int k = 0; k < K; ++k) B[k] = (k == ke_) ? rv : 0.f;
    }

    // Step 1 for a chunk with steps outside [lo, hi), or rows with a period above T (their
    // positions t >= T are skipped): element-wise, masked.
    template <class BaseFn, class PreFn>
    __device__ void load_masked(const Args& a, int64_t lo, int64_t hi, BaseFn&& base_of, int lane,
                                float (&nraw)[Op::kNbrRaw], PreFn&& pre) {
        const int64_t T = a.T, Pd = a.period;
        pre();
        uint32_t inrange = 0;
#pragma unroll
        for (int k = 0; k < K; ++k)
            if (p0 + k >= lo && p0 + k < hi) inrange |= 1u << k;
        valid = 0;
        edge = 0;
#pragma unroll
        for (int k = 0; k < K; ++k) B[k] = 0.f;
        if (inrange) {
            const int64_t first = p0 + __builtin_ctz(inrange);
            int64_t row, t;
            row_and_step(base_of(), first, Pd, a.inv_period, row, t);
#pragma unroll
            for (int k = 0; k < K; ++k) {
                if (p0 + k < first || !bit(inrange, k)) continue;
                if (t < T) {
                    valid |= 1u << k;
                    const bool e = kBack ? (t == T - 1) : (t == 0);
                    if (e) {
                        edge |= 1u << k;
                        if (Op::kRowValue && a.row_value) B[k] = load_one<DT>(a.row_value, row);
                    }
                }
                if (++t == Pd) { t = 0; ++row; }
            }
        }
        term = 0; trunc = 0;
        if (Op::kFlags) {
            if (a.term) term = load_flags_masked<K>(a.term, p0, valid);
            if (TR) trunc = load_flags_masked<K>(a.trunc, p0, valid);
        }
#pragma unroll
        for (int s = 0; s < NS; ++s) {
            if (Op::staged_index(s) >= 0) continue;  // read from LDS in the scan
            if (Op::slot_used(s, TR)) load_k<DT, K>(a.in[s], p0, s == kTS ? (valid & trunc) : valid, false, d[s]);
            else {
#pragma unroll
                for (int k = 0; k < K; ++k) d[s][k] = 0.f;
            }
        }
        if (needs_nbr(lane)) Op::template nbr_load_raw<DT>(a, kBack ? p0 + K : p0 - 1, nraw);
    }

    // Steps 1-4. Writes the wave's map to s_a/s_b[wave] unless `wave_local`; the caller
    // synchronises. Staged policies: `pre` issues the chunk's staging copies (called once the
    // flag loads are out, so that waiting for the flags does not wait for the copies) and `mid`
    // completes the stage (called after every load of the lane is issued, before the staged
    // slots are read).
    template <bool FULL, class BaseFn, class PreFn, class MidFn>
    __device__ void local_scan(const Args& a, int64_t chunk_lo, int64_t lo, int64_t hi,
                               float* s_a, float* s_b, int lane, int wave, bool wave_local,
                               BaseFn&& base_of, const float* staged, PreFn&& pre, MidFn&& mid,
                               float* s_d = nullptr) {
        if constexpr (kCanDefer) {
            defer_chunk_ = FULL && s_d != nullptr && !wave_local;
            defer_ = defer_chunk_ && wave > 0;
        }
        sidx = (wave * kWave + lane_group<kBack>(lane)) * K;
        p0 = chunk_lo + sidx;
        stage = staged;
        float nraw[Op::kNbrRaw];
        if (FULL) load_full(a, lo, hi, base_of, lane, nraw, pre);
        else load_masked(a, lo, hi, base_of, lane, nraw, pre);
        mid();
        if constexpr (Op::kStaged > 0) {
            if (FULL) convert_full(a);
#pragma unroll
            for (int s = 0; s < NS; ++s)
                if (Op::staged_index(s) >= 0) read_staged(s, valid, FULL);
        }

        // Neighbour on the carry-source side of the lane's edge step: lane l-1 holds it, lane 0
        // read it from memory; staged policies read it from the stage (which covers one step
        // past the chunk).
        if constexpr (Op::kStaged > 0) {
            Op::nbr_from_stage(a.p, stage, kStride, kBack ? sidx + K : sidx - 1, nb);
        } else if (Op::kNbr > 0) {
            float own[NB];
            Op::template nbr_export<K>(a.p, d, term | trunc, own);
#pragma unroll
            for (int i = 0; i < NB; ++i) nb[i] = shift_up1(own[i], 0.f);
            if (needs_nbr(lane)) Op::nbr_fix(a, nraw, nb);
        } else {
#pragma unroll
            for (int i = 0; i < NB; ++i) nb[i] = 0.f;
        }

        Op::template build<K, TR>(a.p, d, term, trunc, edge, B, nb, al, be);
        if (!FULL || PAD) {
#pragma unroll
            for (int k = 0; k < K; ++k)
                if (!bit(valid, k)) { al[k] = 0.f; be[k] = 1.f; }
        }

        // Serial composition of the lane's K steps, nearest-to-output outermost.
        Pair agg;
        if (kBack) {
            agg = Pair{al[K - 1], be[K - 1]};
#pragma unroll
            for (int k = K - 2; k >= 0; --k) agg = compose(Pair{al[k], be[k]}, agg);
        } else {
            agg = Pair{al[0], be[0]};
#pragma unroll
            for (int k = 1; k < K; ++k) agg = compose(Pair{al[k], be[k]}, agg);
        }
        incl = wave_scan_inclusive(agg, lane);
        if (!wave_local && lane == kWave - 1) {
            s_a[wave] = incl.a;
            s_b[wave] = incl.b;
            if constexpr (kCanDefer) {
                if (defer_chunk_) s_d[wave] = bit(term | trunc, K - 1) ? 1.f : 0.f;
            }
        }
    }

    // Step 5 (after the barrier): maps of the waves on this wave's carry-source side (and, for
    // a deferring chunk, the cut of each wave's first step by the flag before it).
    __device__ void wave_prefix(const float* s_a, const float* s_b, int wave, const float* s_d = nullptr) {
        Pair acc = identity_pair();
        if (kBack) {
            for (int j = W - 1; j > wave; --j) acc = compose(Pair{s_a[j], s_b[j]}, acc);
        } else {
            // bit j: wave j's last step is done (one LDS read per lane, then scalar bit tests)
            uint64_t done = 0;
            if (kCanDefer && defer_chunk_) {
                const int l = threadIdx.x & (kWave - 1);
                done = __ballot(l < W && s_d[l < W ? l : 0] != 0.f);
            }
            for (int j = 0; j < wave; ++j) {
                const bool cut = kCanDefer && j > 0 && ((done >> (j - 1)) & 1u);
                acc = compose(Pair{s_a[j], cut ? 0.f : s_b[j]}, acc);
            }
            if (kCanDefer && defer_ && ((done >> (wave - 1)) & 1u)) {
                incl.b = 0.f;
                if ((threadIdx.x & (kWave - 1)) == 0) be[0] = 0.f;  // lane 0: the wave's first step
            }
        }
        wave_in = acc;
    }

    // The whole chunk's map (all waves), for publishing.
    __device__ static Pair chunk_map(const float* s_a, const float* s_b) {
        Pair acc = identity_pair();
        if (kBack) {
            for (int j = W - 1; j >= 0; --j) acc = compose(Pair{s_a[j], s_b[j]}, acc);
        } else {
            for (int j = 0; j < W; ++j) acc = compose(Pair{s_a[j], s_b[j]}, acc);
        }
        return acc;
    }

    // Steps 6-7 given the value C just past the chunk on its carry-source side. Returns the
    // value of the lane's step nearest the chunk's output side (A[0] backward, A[K-1] forward).
    template <bool FULL>
    __device__ float finish(const Args& a, float C) {
        const float Xw = apply(wave_in, C);
        // value entering this lane = value leaving lane l-1 on its output side
        const float X = shift_up1(apply(incl, Xw), Xw);
        float A[K];
        if (kBack) {
            float nxt = X;
#pragma unroll
            for (int k = K - 1; k >= 0; --k) { A[k] = fmaf(be[k], nxt, al[k]); nxt = A[k]; }
        } else {
            float prv = X;
#pragma unroll
            for (int k = 0; k < K; ++k) { A[k] = fmaf(be[k], prv, al[k]); prv = A[k]; }
        }
        float o0[K], o1[K];
        Op::template finish<K, TR>(a.p, d, term, trunc, edge, B, nb, A, X, o0, o1);
        const bool vstore = FULL && (!PAD || valid == kAll);
        if constexpr (kLineStores && FULL) {
            if (__all(vstore)) {
                const int lane = threadIdx.x & (kWave - 1);
                const int g = sidx / K - (threadIdx.x / kWave) * kWave;  // the lane's group
                const int64_t base = p0 - int64_t(g) * K;
                store8_lines(a.out0, base, base + kWave * K, g, lane, o0, oslot);
                if (a.out1) store8_lines(a.out1, base, base + kWave * K, g, lane, o1, oslot);
                return kBack ? A[0] : A[K - 1];
            }
        }
        store_k<K>(a.out0, p0, valid, vstore, o0);
        if (a.out1) store_k<K>(a.out1, p0, valid, vstore, o1);
        return kBack ? A[0] : A[K - 1];
    }
};

// One chunk: local scan, the wave composition (unless rows are wave-local) and, through
// `carry_of`, the value entering the chunk; then the carry application and stores.
template <bool FULL, class C, class BaseFn, class CarryFn, class PreFn, class MidFn>
__device__ __forceinline__ float run_chunk(C& c, const Args& a, int64_t chunk_lo, int64_t lo,
                                           int64_t hi, float* s_a, float* s_b, float* s_d,
                                           int lane, int wave, bool wave_local, BaseFn&& base_of,
                                           CarryFn&& carry_of, const float* staged, PreFn&& pre,
                                           MidFn&& mid) {
    c.template local_scan<FULL>(a, chunk_lo, lo, hi, s_a, s_b, lane, wave, wave_local, base_of,
                                staged, pre, mid, s_d);
    if (wave_local) {
        c.wave_in = identity_pair();
    } else {
        __syncthreads();
        c.wave_prefix(s_a, s_b, wave, s_d);
    }
    return c.template finish<FULL>(a, carry_of());
}

// Staging for policies whose per-step terms are reductions over an action axis (full-form
// Retrace). Steps [chunk_lo, chunk_lo + E] that lie in [lo, N*T) are staged (one step past the
// chunk, for the neighbour). `issue` starts copying the chunk's [steps, A] slices of Q (in[1])
// and pi (in[2]) to LDS and loads the steps' actions and behaviour probabilities (in[3]);
// `commit` completes the copies and, after a barrier, the owner thread of each step (steps
// tid, tid + blockDim, ...) reduces its slices into the Op::kStaged staged slots. The caller
// synchronises before the slots are read.
//
// Layout of `dyn` (16-byte aligned): the two slices as DT, `cap` elements each, and, over the
// same bytes once the slices are reduced, kStaged slots of E + 4 floats (the larger of the two is
// the size staged_lds_bytes on the host assumes). With 16-byte aligned
// tensors the 16-byte blocks covering a slice go straight from global memory to LDS
// (global_load_lds_dwordx4: lane l of a wave fills the 16 bytes at the wave-uniform LDS
// address plus 16*l), with no register round trip and every block of the chunk in flight at
// once; LDS element 0 is then the first element of the first block. The one block that can
// reach past the end of the tensors, and the whole slices of unaligned tensors, are copied
// element-wise.
template <class Op, typename DT, int E, int J>
struct Stager {
    static constexpr int64_t kPerBlock = 16 / int64_t(sizeof(DT));
    static constexpr int kStride = E + 4;
    int32_t act[J];
    float mu[J];
    int64_t s_lo, s_hi;      // staged steps
    int64_t el_hi, e0;       // one past the slices' last element; flat element at LDS element 0
    int64_t el_copy;         // elements [el_copy, el_hi) are copied element-wise

    __device__ static int64_t cap(int64_t A) {
        return ((int64_t(E + 1) * A + 3 * kPerBlock) / kPerBlock) * kPerBlock;
    }

    __device__ __forceinline__ void issue(const Args& a, int64_t chunk_lo, int64_t lo, float* dyn) {
        const int64_t total = a.N * a.T, A = a.A;
        const int nt = blockDim.x, tid = threadIdx.x;
        s_lo = max(chunk_lo, lo);
        s_hi = max(min(chunk_lo + E + 1, total), s_lo);
        // unconditional loads from a clamped step (s_lo is in range), so that no branch waits
        // for them
#pragma unroll
        for (int j = 0; j < J; ++j) {
            const int64_t i = tid + int64_t(j) * nt;  // stage index
            const int64_t st = chunk_lo + i;
            const bool ok = i <= E && st >= s_lo && st < s_hi;
            const int64_t sc = ok ? st : s_lo;
            const int32_t act_raw = a.actions[sc];
            const float mu_raw = load_one<DT>(a.in[3], sc);
            act[j] = ok ? act_raw : -1;
            mu[j] = ok ? mu_raw : 1.f;
        }
        const int64_t el_lo = s_lo * A;
        el_hi = s_hi * A;
        if (!a.stage_vec) {
            e0 = el_lo;
            el_copy = el_lo;
            return;
        }
        const int64_t blk_lo = el_lo / kPerBlock;
        const int64_t nblk = el_hi > el_lo ? (el_hi + kPerBlock - 1) / kPerBlock - blk_lo : 0;
        const int64_t nfull = min(nblk, max(total * A / kPerBlock - blk_lo, int64_t(0)));
        e0 = blk_lo * kPerBlock;
        el_copy = max(el_lo, (blk_lo + nfull) * kPerBlock);
        const u32x4* gq = reinterpret_cast<const u32x4*>(a.in[1]) + blk_lo;
        const u32x4* gp = reinterpret_cast<const u32x4*>(a.in[2]) + blk_lo;
        u32x4* lq = reinterpret_cast<u32x4*>(dyn);
        u32x4* lp = lq + cap(A) / kPerBlock;
        const int lane = tid & (kWave - 1);
        for (int64_t b0 = tid - lane; b0 < nfull; b0 += nt) {
            if (b0 + lane < nfull) {
                __builtin_amdgcn_global_load_lds(gq + b0 + lane, (__attribute__((address_space(3))) void*)(lq + b0), 16, 0, 0);
                __builtin_amdgcn_global_load_lds(gp + b0 + lane, (__attribute__((address_space(3))) void*)(lp + b0), 16, 0, 0);
            }
        }
    }

    __device__ __forceinline__ void commit(const Args& a, int64_t chunk_lo, float* dyn) {
        const int64_t A = a.A;
        const int nt = blockDim.x, tid = threadIdx.x;
        DT* sq = reinterpret_cast<DT*>(dyn);
        DT* sp = sq + cap(A);
        const DT* gq = reinterpret_cast<const DT*>(a.in[1]);
        const DT* gp = reinterpret_cast<const DT*>(a.in[2]);
        const int64_t n_el = el_hi - el_copy;
        for (int64_t base = tid; base < n_el; base += 8 * int64_t(nt)) {
            DT vq[8], vp[8];
#pragma unroll
            for (int u = 0; u < 8; ++u) {
                const int64_t m = base + int64_t(u) * nt;
                if (m < n_el) { vq[u] = gq[el_copy + m]; vp[u] = gp[el_copy + m]; }
            }
#pragma unroll
            for (int u = 0; u < 8; ++u) {
                const int64_t m = base + int64_t(u) * nt;
                if (m < n_el) { sq[el_copy - e0 + m] = vq[u]; sp[el_copy - e0 + m] = vp[u]; }
            }
        }
        // the LDS copies of this wave have landed; then every wave's have
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
        __syncthreads();
        // rows are 16-byte aligned whole blocks in LDS when A is a multiple of a block
        const bool rows16 = a.stage_vec && A % kPerBlock == 0;
        float v[J][Op::kStaged];
        bool bad = false;
#pragma unroll
        for (int j = 0; j < J; ++j) {
            const int64_t i = tid + int64_t(j) * nt;
            const int64_t st = chunk_lo + i;
#pragma unroll
            for (int q = 0; q < Op::kStaged; ++q) v[j][q] = 0.f;
            if (i <= E && st >= s_lo && st < s_hi) {
                Op::template reduce_step<DT>(sq + (st * A - e0), sp + (st * A - e0), A, rows16, act[j], mu[j], v[j]);
                bad = bad || act[j] < 0 || act[j] >= A;
            }
        }
        if (bad && a.ws) report_bad_action(a.ws);
        // the slots overlay the slices: every slice read is done before any slot is written
        __syncthreads();
#pragma unroll
        for (int j = 0; j < J; ++j) {
            const int64_t i = tid + int64_t(j) * nt;
            if (i > E) continue;
#pragma unroll
            for (int q = 0; q < Op::kStaged; ++q) dyn[q * kStride + i] = v[j][q];
        }
    }
};

// Staging for action axes too long for a chunk's whole [steps, A] slices in LDS: the axis is
// taken in slices of a.A_slice actions (whole 128-byte lines of DT where one fits, else a
// multiple of 16 bytes). For each slice, the [staged steps, slice] blocks of Q and pi go to
// LDS (row stride = the slice's width: by
// global_load_lds_dwordx4 when every row segment is whole aligned 16-byte blocks, element-wise
// otherwise), and the owner thread of each step adds the slice's terms to its running sums:
// E_pi Q over the actions in order (the same sequence of fused multiply-adds as one slice
// holding the whole axis), and Q and pi of the taken action when it lies in the slice. A
// barrier separates each slice's reads from the next slice's copies, and the last reads from
// the slots, which overlay the slices as in Stager. The first slice is issued with the chunk's
// other loads; the others follow one at a time.
template <class Op, typename DT, int E, int J>
struct SlicedStager {
    static constexpr int64_t kPerBlock = 16 / int64_t(sizeof(DT));
    static constexpr int kStride = E + 4;
    int32_t act[J];
    float mu[J];
    float qa[J], ex[J], pa[J];
    int64_t s_lo, s_hi;

    // LDS elements of one array's slab of `As` actions (rounded up to whole 16-byte blocks).
    __device__ static int64_t cap(int64_t As) {
        return (int64_t(E + 1) * As + kPerBlock - 1) / kPerBlock * kPerBlock;
    }

    __device__ __forceinline__ void copy_slice(const Args& a, int64_t a0, int64_t aw, float* dyn) {
        const int64_t A = a.A, rows = s_hi - s_lo;
        const int nt = blockDim.x, tid = threadIdx.x;
        DT* sq = reinterpret_cast<DT*>(dyn);
        DT* sp = sq + cap(a.A_slice);
        if (a.stage_vec && A % kPerBlock == 0 && aw % kPerBlock == 0) {
            // a0 is a multiple of the slice width, itself a multiple of kPerBlock
            const int64_t bpr = aw / kPerBlock, nblk = rows * bpr;
            const u32x4* gq = reinterpret_cast<const u32x4*>(a.in[1]);
            const u32x4* gp = reinterpret_cast<const u32x4*>(a.in[2]);
            u32x4* lq = reinterpret_cast<u32x4*>(sq);
            u32x4* lp = reinterpret_cast<u32x4*>(sp);
            const int lane = tid & (kWave - 1);
            for (int64_t b0 = tid - lane; b0 < nblk; b0 += nt) {
                const int64_t b = b0 + lane;
                if (b < nblk) {
                    const int64_t row = b / bpr, cb = b - row * bpr;
                    const int64_t g = ((s_lo + row) * A + a0) / kPerBlock + cb;
                    __builtin_amdgcn_global_load_lds(gq + g, (__attribute__((address_space(3))) void*)(lq + b0), 16, 0, 0);
                    __builtin_amdgcn_global_load_lds(gp + g, (__attribute__((address_space(3))) void*)(lp + b0), 16, 0, 0);
                }
            }
        } else {
            const DT* gq = reinterpret_cast<const DT*>(a.in[1]);
            const DT* gp = reinterpret_cast<const DT*>(a.in[2]);
            for (int64_t row = tid / aw, c = tid % aw; row < rows;) {
                const int64_t g = (s_lo + row) * A + a0 + c;
                sq[row * aw + c] = gq[g];
                sp[row * aw + c] = gp[g];
                c += nt;
                row += c / aw;
                c %= aw;
            }
        }
    }

    __device__ __forceinline__ void issue(const Args& a, int64_t chunk_lo, int64_t lo, float* dyn) {
        const int64_t total = a.N * a.T;
        const int nt = blockDim.x, tid = threadIdx.x;
        s_lo = max(chunk_lo, lo);
        s_hi = max(min(chunk_lo + E + 1, total), s_lo);
#pragma unroll
        for (int j = 0; j < J; ++j) {
            const int64_t i = tid + int64_t(j) * nt;  // stage index
            const int64_t st = chunk_lo + i;
            const bool ok = i <= E && st >= s_lo && st < s_hi;
            const int64_t sc = ok ? st : s_lo;
            const int32_t act_raw = a.actions[sc];
            const float mu_raw = load_one<DT>(a.in[3], sc);
            act[j] = ok ? act_raw : -1;
            mu[j] = ok ? mu_raw : 1.f;
            qa[j] = ex[j] = pa[j] = 0.f;
        }
        copy_slice(a, 0, min(a.A_slice, a.A), dyn);
    }

    __device__ __forceinline__ void commit(const Args& a, int64_t chunk_lo, float* dyn) {
        const int64_t A = a.A, As = a.A_slice;
        const int nt = blockDim.x, tid = threadIdx.x;
        const DT* sq = reinterpret_cast<const DT*>(dyn);
        const DT* sp = sq + cap(As);
        for (int64_t a0 = 0;;) {
            const int64_t aw = min(As, A - a0);
            // the LDS copies of this wave have landed; then every wave's have
            asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
            __syncthreads();
#pragma unroll
            for (int j = 0; j < J; ++j) {
                const int64_t i = tid + int64_t(j) * nt;
                const int64_t st = chunk_lo + i;
                if (i <= E && st >= s_lo && st < s_hi)
                    Op::template accumulate_slice<DT>(sq + (st - s_lo) * aw, sp + (st - s_lo) * aw, a0, aw,
                                                      act[j], ex[j], qa[j], pa[j]);
            }
            a0 += aw;
            if (a0 >= A) break;
            __syncthreads();  // every read of this slice is done before the next one lands
            copy_slice(a, a0, min(As, A - a0), dyn);
        }
        // the slots overlay the slices: every slice read is done before any slot is written
        __syncthreads();
        bool bad = false;
#pragma unroll
        for (int j = 0; j < J; ++j) {
            const int64_t i = tid + int64_t(j) * nt;
            if (i > E) continue;
            const int64_t st = chunk_lo + i;
            const bool in = st >= s_lo && st < s_hi;
            bad = bad || (in && (act[j] < 0 || act[j] >= A));
            float v[Op::kStaged] = {in ? qa[j] : 0.f, in ? ex[j] : 0.f, in ? pa[j] / mu[j] : 0.f};
#pragma unroll
            for (int q = 0; q < Op::kStaged; ++q) dyn[q * kStride + i] = v[q];
        }
        if (bad && a.ws) report_bad_action(a.ws);
    }
};

// Policies without staging.
template <class Op, typename DT, int E, int J>
struct NoStager {
    __device__ void issue(const Args&, int64_t, int64_t, float*) {}
    __device__ void commit(const Args&, int64_t, float*) {}
};

// Rows kernel: workgroup g owns rows [g*R, g*R + R) and walks them in chunks of E steps
// aligned to multiples of K, starting from the carry source (the end for backward scans).
// `wave_local`: every wave's span starts and ends on row edges (T divides 64*K and the chunk
// is row aligned), so no carry crosses waves and step 5 is skipped.
template <class Op, typename DT, int K, int W, bool VEC, bool TR, bool PAD = false>
__global__ void __launch_bounds__(W * kWave) rows_kernel(Args a, int64_t rows_per_wg, int wave_local) {
    using C = Chunk<Op, DT, K, W, VEC, TR, PAD>;
    constexpr int64_t E = int64_t(W) * kWave * K;
    using S = std::conditional_t<(Op::kStaged > 0),
                                 std::conditional_t<Op::kSliced, SlicedStager<Op, DT, int(E), K + 1>,
                                                    Stager<Op, DT, int(E), K + 1>>,
                                 NoStager<Op, DT, int(E), K + 1>>;
    __shared__ float s_a[W], s_b[W];
    __shared__ float s_d[C::kCanDefer ? W : 1];
    __shared__ float s_carry;
    __shared__ f32x4 s_out[C::kLineStores ? W : 1][C::kLineStores ? 2 * kWave : 1];
    const int lane = threadIdx.x & (kWave - 1), wave = threadIdx.x / kWave;
    const int64_t row_lo = int64_t(blockIdx.x) * rows_per_wg;
    const int64_t row_hi = min(row_lo + rows_per_wg, a.N);
    // the range ends at the last row's last step (rows lie `period` apart; its gap is not part)
    const int64_t lo = row_lo * a.period, hi = (row_hi - 1) * a.period + a.T;
    const bool can_full = VEC && a.T >= K && (PAD || a.period == a.T);
    float carry = 0.f;
    auto carry_of = [&]() { return carry; };
    extern __shared__ __align__(16) float s_dyn[];  // staged policies only (sized at launch)
    const float* stage = Op::kStaged > 0 ? s_dyn : nullptr;
    // the workgroup's first step is the start of row row_lo
    auto base_of = [&]() { return RowBase{lo, row_lo, 0}; };
    if (Op::kBackward) {
        int64_t chunk_hi = (hi + K - 1) / K * K;
        for (;;) {
            const int64_t chunk_lo = chunk_hi - E;
            S sg;
            auto pre = [&]() { sg.issue(a, chunk_lo, lo, s_dyn); };
            auto mid = [&]() { if constexpr (Op::kStaged > 0) { sg.commit(a, chunk_lo, s_dyn); __syncthreads(); } };
            C c;
            c.oslot = s_out[C::kLineStores ? wave : 0];
            const float first = (can_full && (PAD || (chunk_lo >= lo && chunk_hi <= hi)))
                ? run_chunk<true>(c, a, chunk_lo, lo, hi, s_a, s_b, s_d, lane, wave, wave_local, base_of, carry_of, stage, pre, mid)
                : run_chunk<false>(c, a, chunk_lo, lo, hi, s_a, s_b, s_d, lane, wave, wave_local, base_of, carry_of, stage, pre, mid);
            if (chunk_lo <= lo) break;
            // the next chunk (earlier in time) continues from A at chunk_lo, held by lane 63 of
            // wave 0
            if (threadIdx.x == kWave - 1) s_carry = first;
            __syncthreads();
            carry = s_carry;
            chunk_hi = chunk_lo;
        }
    } else {
        int64_t chunk_lo = lo / K * K;
        for (;;) {
            S sg;
            auto pre = [&]() { sg.issue(a, chunk_lo, lo, s_dyn); };
            auto mid = [&]() { if constexpr (Op::kStaged > 0) { sg.commit(a, chunk_lo, s_dyn); __syncthreads(); } };
            C c;
            c.oslot = s_out[C::kLineStores ? wave : 0];
            const float last = (can_full && (PAD || (chunk_lo >= lo && chunk_lo + E <= hi)))
                ? run_chunk<true>(c, a, chunk_lo, lo, hi, s_a, s_b, s_d, lane, wave, wave_local, base_of, carry_of, stage, pre, mid)
                : run_chunk<false>(c, a, chunk_lo, lo, hi, s_a, s_b, s_d, lane, wave, wave_local, base_of, carry_of, stage, pre, mid);
            if (chunk_lo + E >= hi) break;
            if (threadIdx.x == W * kWave - 1) s_carry = last;
            __syncthreads();
            carry = s_carry;
            chunk_lo += E;
        }
    }
}

// Rows that tile a wave exactly: T a power of two with K <= T <= 64*K, dense rows, every array
// aligned for the vector path. One wave per workgroup; wave g owns steps [g*64*K, (g+1)*64*K)
// of the flat [N*T] array, lane l the l-th group of K steps (the (63-l)-th backward), so every
// row lies inside one wave and its edge step inside one lane. A lane's row and step are a
// shift and a mask of its position, and the step after (before) the lane's last (first) one
// is either in lane l-1 or across the row's edge, so no neighbour is read from memory and
// nothing crosses waves: per lane, the flag words, the data vectors and the per-row value are
// issued back to back, the continuation vector follows only where a step is truncated, then
// Table 1's coefficients, the lane's serial map, the DPP wave scan and the stores. Lanes past
// the array's end (its last wave may be partial; N*T is a multiple of K) load step 0 of row
// 0 and store nothing. The WPG waves of a workgroup take consecutive wave spans, each on its
// own (no LDS, no barrier). Grid: ceil(N*T / (64*K*WPG)) workgroups of WPG waves.
template <class Op, typename DT, int K, bool TR, int WPG = 1>
__global__ void __launch_bounds__(WPG * kWave) wave_rows_kernel(Args a, int log2T) {
    static_assert(Op::kStaged == 0, "staged policies run on the rows kernel");
    constexpr bool kBack = Op::kBackward;
    constexpr int NS = Op::kSlots;
    constexpr int NB = Op::kNbr > 0 ? Op::kNbr : 1;
    constexpr int kWords = K * int(sizeof(DT)) / 4;
    constexpr int kTS = TR ? Op::kTruncSlot : -1;
    const int lane = threadIdx.x & (kWave - 1);
    const int64_t T = a.T;
    const int64_t p0 = (int64_t(blockIdx.x) * WPG + threadIdx.x / kWave) * (kWave * K) +
                       int64_t(lane_group<kBack>(lane)) * K;
    const bool live = p0 < a.N * T;
    const int64_t pc = live ? p0 : 0;
    const uint8_t* fallback = reinterpret_cast<const uint8_t*>(a.in[0]);

    uint32_t tw[(K + 3) / 4], rw[(K + 3) / 4];
    uint32_t w[NS][kWords];
    if (Op::kFlags && TR) load_flag_words<K>(a.trunc, pc, rw);
    if (Op::kFlags) load_flag_words<K>(a.term ? a.term : fallback, pc, tw);
#pragma unroll
    for (int s = 0; s < NS; ++s)
        if (Op::slot_used(s, TR) && s != kTS) load_words<DT, K>(a.in[s], pc, w[s]);
    const int64_t row = pc >> log2T;
    const int64_t t = pc & (T - 1);
    const bool has_rv = Op::kRowValue && a.row_value;
    const float rv = load_one<DT>(has_rv ? a.row_value : a.in[0], row);
    // the row's edge step, if among the lane's K steps (T is a multiple of K)
    const int ke = kBack ? (t + K == T ? K - 1 : -1) : (t == 0 ? 0 : -1);
    const uint32_t edge = ke >= 0 ? (1u << ke) : 0u;
    const uint32_t trunc = (Op::kFlags && TR) ? flag_mask<K>(rw) : 0u;
    if constexpr (kTS >= 0) {
        if (trunc) load_words<DT, K>(a.in[kTS], pc, w[kTS]);
        else {
#pragma unroll
            for (int i = 0; i < kWords; ++i) w[kTS][i] = 0u;
        }
    }
    float d[NS][K];
#pragma unroll
    for (int s = 0; s < NS; ++s) {
        if (Op::slot_used(s, TR)) unpack_words<DT, K>(w[s], d[s]);
        else {
#pragma unroll
            for (int k = 0; k < K; ++k) d[s][k] = 0.f;
        }
    }
    const uint32_t term = (Op::kFlags && a.term) ? flag_mask<K>(tw) : 0u;
    float B[K];
#pragma unroll
    for (int k = 0; k < K; ++k) B[k] = (k == ke && has_rv) ? rv : 0.f;

    // neighbour on the carry-source side: lane l-1 (across a row edge it is not used)
    float nb[NB];
    if constexpr (Op::kNbr > 0) {
        float own[NB];
        Op::template nbr_export<K>(a.p, d, term | trunc, own);
#pragma unroll
        for (int i = 0; i < NB; ++i) nb[i] = shift_up1(own[i], 0.f);
    } else {
#pragma unroll
        for (int i = 0; i < NB; ++i) nb[i] = 0.f;
    }
    float al[K], be[K];
    Op::template build<K, TR>(a.p, d, term, trunc, edge, B, nb, al, be);
    if (!live) {
#pragma unroll
        for (int k = 0; k < K; ++k) { al[k] = 0.f; be[k] = 1.f; }
    }
    Pair agg;
    if (kBack) {
        agg = Pair{al[K - 1], be[K - 1]};
#pragma unroll
        for (int k = K - 2; k >= 0; --k) agg = compose(Pair{al[k], be[k]}, agg);
    } else {
        agg = Pair{al[0], be[0]};
#pragma unroll
        for (int k = 1; k < K; ++k) agg = compose(Pair{al[k], be[k]}, agg);
    }
    const Pair incl = wave_scan_inclusive(agg, lane);
    // value entering this lane: the value leaving lane l-1 (nothing enters lane 0, whose
    // carry-source side is a row edge)
    const float X = shift_up1(incl.a, 0.f);
    float A[K];
    if (kBack) {
        float nxt = X;
#pragma unroll
        for (int k = K - 1; k >= 0; --k) { A[k] = fmaf(be[k], nxt, al[k]); nxt = A[k]; }
    } else {
        float prv = X;
#pragma unroll
        for (int k = 0; k < K; ++k) { A[k] = fmaf(be[k], prv, al[k]); prv = A[k]; }
    }
    float o0[K], o1[K];
    Op::template finish<K, TR>(a.p, d, term, trunc, edge, B, nb, A, X, o0, o1);
    if constexpr (K == 8) {
        // the wave's outputs are [base, base + 512): whole-line stores through LDS
        __shared__ f32x4 s_out[WPG][2 * kWave];
        f32x4* slot = s_out[threadIdx.x / kWave];
        const int g = lane_group<kBack>(lane);
        const int64_t base = p0 - int64_t(g) * K, limit = a.N * T;
        store8_lines(a.out0, base, limit, g, lane, o0, slot);
        if (a.out1) store8_lines(a.out1, base, limit, g, lane, o1, slot);
    } else if (live) {
        store_k<K>(a.out0, p0, 0u, true, o0);
        if (a.out1) store_k<K>(a.out1, p0, 0u, true, o1);
    }
}

// Dense rows, K < T <= W*64*K: workgroup g owns rows [g*R, g*R + R), R*T <= W*64*K and a
// multiple of K (and N*T a multiple of K), one contiguous, vector-aligned range [lo, hi); a row
// edge may fall inside a lane's K steps when T is not a multiple of K. Its W*64 lanes take
// consecutive groups of K steps from lo (the (63-l)-th group of each wave backward), the lanes
// past hi idle and loading nothing. Rows may straddle waves but not workgroups: each wave scans
// its lanes as wave_rows_kernel does, the waves compose through LDS once, and lane 0 of a wave
// reads its carry-source neighbour from memory with its other loads (it lies in the next or
// previous wave's span unless a row edge comes first). A lane's row and step come from its
// offset q in the range by a multiply and a shift: floor(q * magic / 2^s) = floor(q / T) with
// magic = ceil(2^s / T), since q * (magic - 2^s / T) / 2^s < 1 / T whenever q * T < 2^s:
// s = flat_shift(W), 22 for four waves (q < 1024 fp32 or 2048 bf16 steps, T below 2048) and
// 26 for sixteen (q < 4096 fp32 steps, T up to 4096), with q * magic below 2^32 (the host
// takes sixteen waves only for rows of more than 256 steps). No chunk loop, no element-wise
// path. Grid: ceil(N / R) workgroups.
constexpr int flat_shift(int W) { return W > 4 ? 26 : 22; }

template <class Op, typename DT, int K, bool TR, int W>
__global__ void __launch_bounds__(W * kWave) flat_rows_kernel(Args a, int R, uint32_t magic) {
    static_assert(Op::kStaged == 0, "staged policies run on the rows kernel");
    constexpr bool kBack = Op::kBackward;
    constexpr int NS = Op::kSlots;
    constexpr int NB = Op::kNbr > 0 ? Op::kNbr : 1;
    constexpr int kWords = K * int(sizeof(DT)) / 4;
    constexpr int kTS = TR ? Op::kTruncSlot : -1;
    __shared__ float s_a[W], s_b[W];
    const int lane = threadIdx.x & (kWave - 1), wave = threadIdx.x / kWave;
    const int64_t T = a.T;
    const int64_t row0 = int64_t(blockIdx.x) * R;
    const int64_t lo = row0 * T;
    const int64_t hi = min(row0 + R, a.N) * T;
    const int g = lane_group<kBack>(lane);
    const int q = (wave * kWave + g) * K;  // the lane's offset in the range
    const int64_t p0 = lo + q;
    const bool live = p0 < hi;
    const int64_t pc = live ? p0 : 0;
    const uint8_t* fallback = reinterpret_cast<const uint8_t*>(a.in[0]);

    // Idle lanes load nothing: all of them reading one clamped address would pile every
    // workgroup's idle loads onto a single line.
    uint32_t tw[(K + 3) / 4] = {}, rw[(K + 3) / 4] = {};
    uint32_t w[NS][kWords] = {};
    float nraw[Op::kNbrRaw] = {};
    if (live) {
        if (Op::kFlags && TR) load_flag_words<K>(a.trunc, pc, rw);
        if (Op::kFlags) load_flag_words<K>(a.term ? a.term : fallback, pc, tw);
#pragma unroll
        for (int s = 0; s < NS; ++s)
            if (Op::slot_used(s, TR) && s != kTS) load_words<DT, K>(a.in[s], pc, w[s]);
        // lane 0: the step past its carry-source edge, from memory (used unless a row edge
        // comes first; an address outside the range is replaced by the lane's own)
        if constexpr (Op::kNbr > 0) {
            const int64_t pn = kBack ? p0 + K : p0 - 1;
            const bool in = kBack ? pn < hi : pn >= lo;
            if (lane == 0) Op::template nbr_load_raw<DT>(a, in ? pn : pc, nraw);
        }
    }
    const int r_in = int((uint32_t(q) * magic) >> flat_shift(W));
    const int64_t row = live ? row0 + r_in : 0;
    const int64_t t = live ? int64_t(q - r_in * int(T)) : 0;
    // the row edge among the lane's K steps, if any (at most one: T >= K): backward the last
    // step of the lane's first row, forward the first step of a row (the next one when the
    // lane starts inside a row)
    int ke = -1;
    if (kBack) {
        if (t + K >= T) ke = int(T - 1 - t);
    } else {
        if (t == 0) ke = 0;
        else if (t + K > T) ke = int(T - t);
    }
    const uint32_t edge = (live && ke >= 0) ? (1u << ke) : 0u;
    // the per-row value belongs to the edge's row: forward, a row starting inside the lane is
    // the next one (it lies in the range, so it exists)
    const int64_t row_e = (!kBack && ke > 0) ? row + 1 : row;
    const bool has_rv = Op::kRowValue && a.row_value;
    const float rv = (has_rv && live) ? load_one<DT>(a.row_value, row_e) : 0.f;
    const uint32_t trunc = (Op::kFlags && TR) ? flag_mask<K>(rw) : 0u;
    if constexpr (kTS >= 0) {
        if (trunc) load_words<DT, K>(a.in[kTS], pc, w[kTS]);
        else {
#pragma unroll
            for (int i = 0; i < kWords; ++i) w[kTS][i] = 0u;
        }
    }
    float d[NS][K];
#pragma unroll
    for (int s = 0; s < NS; ++s) {
        if (Op::slot_used(s, TR)) unpack_words<DT, K>(w[s], d[s]);
        else {
#pragma unroll
            for (int k = 0; k < K; ++k) d[s][k] = 0.f;
        }
    }
    const uint32_t term = (Op::kFlags && a.term) ? flag_mask<K>(tw) : 0u;
    float B[K];
#pragma unroll
    for (int k = 0; k < K; ++k) B[k] = (k == ke && has_rv) ? rv : 0.f;

    // neighbour on the carry-source side: lane l-1, or for lane 0 the step read from memory
    float nb[NB];
    if constexpr (Op::kNbr > 0) {
        float own[NB];
        Op::template nbr_export<K>(a.p, d, term | trunc, own);
#pragma unroll
        for (int i = 0; i < NB; ++i) nb[i] = shift_up1(own[i], 0.f);
        if (lane == 0 && live && !(edge & (kBack ? (1u << (K - 1)) : 1u))) Op::nbr_fix(a, nraw, nb);
    } else {
#pragma unroll
        for (int i = 0; i < NB; ++i) nb[i] = 0.f;
    }
    float al[K], be[K];
    Op::template build<K, TR>(a.p, d, term, trunc, edge, B, nb, al, be);
    if (!live) {
#pragma unroll
        for (int k = 0; k < K; ++k) { al[k] = 0.f; be[k] = 1.f; }
    }
    Pair agg;
    if (kBack) {
        agg = Pair{al[K - 1], be[K - 1]};
#pragma unroll
        for (int k = K - 2; k >= 0; --k) agg = compose(Pair{al[k], be[k]}, agg);
    } else {
        agg = Pair{al[0], be[0]};
#pragma unroll
        for (int k = 1; k < K; ++k) agg = compose(Pair{al[k], be[k]}, agg);
    }
    const Pair incl = wave_scan_inclusive(agg, lane);
    // the waves on this wave's carry-source side, composed (the range's carry-source end is a
    // row edge, so nothing enters the range)
    if (lane == kWave - 1) { s_a[wave] = incl.a; s_b[wave] = incl.b; }
    __syncthreads();
    Pair win = identity_pair();
    if (kBack) {
        for (int j = W - 1; j > wave; --j) win = compose(Pair{s_a[j], s_b[j]}, win);
    } else {
        for (int j = 0; j < wave; ++j) win = compose(Pair{s_a[j], s_b[j]}, win);
    }
    const float Xw = win.a;
    const float X = shift_up1(apply(incl, Xw), Xw);
    float A[K];
    if (kBack) {
        float nxt = X;
#pragma unroll
        for (int k = K - 1; k >= 0; --k) { A[k] = fmaf(be[k], nxt, al[k]); nxt = A[k]; }
    } else {
        float prv = X;
#pragma unroll
        for (int k = 0; k < K; ++k) { A[k] = fmaf(be[k], prv, al[k]); prv = A[k]; }
    }
    float o0[K], o1[K];
    Op::template finish<K, TR>(a.p, d, term, trunc, edge, B, nb, A, X, o0, o1);
    if constexpr (K == 8) {
        // the wave's outputs are [base, base + 512) up to hi: stores of 16-byte pieces in order
        __shared__ f32x4 s_out[W][2 * kWave];
        const int64_t base = lo + int64_t(wave) * kWave * K;
        store8_lines(a.out0, base, hi, g, lane, o0, s_out[wave]);
        if (a.out1) store8_lines(a.out1, base, hi, g, lane, o1, s_out[wave]);
    } else if (live) {
        store_k<K>(a.out0, p0, 0u, true, o0);
        if (a.out1) store_k<K>(a.out1, p0, 0u, true, o1);
    }
}

// Polls of one record before a waiting tile gives up (about a second). Reached only when the
// workspace was not zero-filled before first use; the tile then continues with a NaN carry
// and flags the workspace header instead of waiting forever.
constexpr uint32_t kMaxPolls = 1u << 20;

// Value entering tile `tile` of a row from its carry-source side, composed from the published
// maps of the row's other tiles (tile q's record at rec_row + q * rstride), nearest outermost;
// run by one full wave. Lane l looks at the tile 63-l places further (so the nearest tile sits
// in lane 63, outermost in the prefix scan).
template <bool kBack>
__device__ float gather_carry(const uint64_t* rec_row, int64_t rstride, int64_t tile, int64_t P,
                              uint32_t tag0, uint32_t tag1, int lane, WsHeader* hdr) {
    const int dist = kWave - 1 - lane;
    Pair acc = identity_pair();
    int64_t step = 1;
    for (;;) {
        const int64_t j = kBack ? tile + step + dist : tile - step - dist;
        const bool inside = kBack ? (j < P) : (j >= 0);
        Pair v = Pair{0.f, 0.f};  // past the row edge: nothing flows in
        bool ready = !inside;
        uint64_t prefix_mask, sever_mask;
        for (uint32_t polls = 0;; ++polls) {
            if (!ready) {
                const uint64_t w0 = ld_relaxed(rec_row + j * rstride);
                const uint64_t w1 = ld_relaxed(rec_row + j * rstride + 1);
                if (uint32_t(w0 >> 32) == tag0 && uint32_t(w1 >> 32) == tag1) {
                    ready = true;
                    v = Pair{__uint_as_float(uint32_t(w0)), __uint_as_float(uint32_t(w1))};
                }
            }
            const uint64_t rmask = __ballot(ready);
            sever_mask = __ballot(ready && v.b == 0.f);
            // ready tiles counted from the nearest (lane 63) down
            const int run = (rmask == ~0ull) ? 64 : __builtin_clzll(~rmask);
            prefix_mask = (run == 64) ? ~0ull : ~((~0ull) >> run);
            if ((sever_mask & prefix_mask) != 0ull || run == 64) break;
            if (polls >= kMaxPolls) {
                if (lane == 0) st_relaxed(&hdr->error, 1u);
                return __builtin_nanf("");
            }
            __builtin_amdgcn_s_sleep(1);
        }
        const uint64_t sev = sever_mask & prefix_mask;
        const int stop = sev ? __builtin_clzll(sev) : 64;  // distance of the nearest sever
        const Pair mine = (dist <= stop) ? v : identity_pair();
        const Pair batch = read_lane(wave_scan_inclusive(mine, lane), kWave - 1);
        acc = compose(acc, batch);
        if (stop < 64) return acc.a;
        step += kWave;
    }
}

// Tiles kernel: row n split into P tiles of E steps (the last one may be shorter), one
// workgroup per tile, carries passed through the workspace. Workgroup g serves row g mod N and
// takes its tile from that row's ticket, in carry-source order. Grid = N * P (N <= kWsSlots).
template <class Op, typename DT, int K, int W, bool VEC, bool TR>
__global__ void __launch_bounds__(W * kWave) tiles_kernel(Args a, int64_t P) {
    using C = Chunk<Op, DT, K, W, VEC, TR>;
    constexpr bool kBack = Op::kBackward;
    constexpr int64_t E = int64_t(W) * kWave * K;
    __shared__ float s_a[W], s_b[W];
    __shared__ float s_carry;
    __shared__ uint32_t s_ticket, s_gen;
    __shared__ f32x4 s_out[C::kLineStores ? W : 1][C::kLineStores ? 2 * kWave : 1];
    WsHeader* hdr = reinterpret_cast<WsHeader*>(a.ws);
    uint64_t* rec = reinterpret_cast<uint64_t*>(reinterpret_cast<char*>(a.ws) + kWsRecordsOffset);
    const int lane = threadIdx.x & (kWave - 1), wave = threadIdx.x / kWave;
    const int64_t N = a.N, T = a.T;
    const int64_t row = int64_t(blockIdx.x) % N;

    if (threadIdx.x == 0) {
        uint32_t gen;
        s_ticket = draw_ticket(draw_word(a.ws, row), P, gen);
        s_gen = gen;
    }
    __syncthreads();
    const uint32_t tag0 = 2u * s_gen + 1u;
    const uint32_t tag1 = tag0 + uint32_t(N) * kTagMix;
    const int64_t ticket = s_ticket;
    if (wave == 0) advance_idle_slots(a.ws, N, s_gen, lane);
    if (ticket >= P) {
        // Only possible if the workspace was not zero-filled before first use.
        if (threadIdx.x == 0) st_relaxed(&hdr->error, 1u);
        return;
    }
    const int64_t p = kBack ? P - 1 - ticket : ticket;
    const int64_t lo = row * T + p * E, hi = min(lo + E, row * T + T);

    C c;
    c.oslot = s_out[C::kLineStores ? wave : 0];
    // whole 16-byte vectors: a full tile whose rows start on a vector boundary
    const bool full = VEC && T % K == 0 && hi - lo == E;
    auto base_of = [&]() { return RowBase{lo, row, p * E}; };
    static_assert(Op::kStaged == 0, "staged policies run on the rows kernel only");
    if (full) c.template local_scan<true>(a, lo, lo, hi, s_a, s_b, lane, wave, false, base_of, nullptr, Nop{}, Nop{});
    else c.template local_scan<false>(a, lo, lo, hi, s_a, s_b, lane, wave, false, base_of, nullptr, Nop{}, Nop{});
    __syncthreads();
    c.wave_prefix(s_a, s_b, wave);

    // A tile is read by its neighbour on the output side unless it holds the row's output-side
    // edge; it needs a carry unless it holds the row's carry-source edge.
    const bool publish = kBack ? (p > 0) : (p < P - 1);
    const bool need = kBack ? (p < P - 1) : (p > 0);
    if (publish && threadIdx.x == 0) {
        const Pair m = C::chunk_map(s_a, s_b);
        st_relaxed(rec + 2 * (p * N + row), uint64_t(tag0) << 32 | __float_as_uint(m.a));
        st_relaxed(rec + 2 * (p * N + row) + 1, uint64_t(tag1) << 32 | __float_as_uint(m.b));
    }
    if (need && wave == 0) {
        const float v = gather_carry<kBack>(rec + 2 * row, 2 * N, p, P, tag0, tag1, lane, hdr);
        if (lane == 0) s_carry = v;
    }
    __syncthreads();
    const float carry = need ? s_carry : 0.f;
    if (full) c.template finish<true>(a, carry);
    else c.template finish<false>(a, carry);
}

}  // namespace rlcs
