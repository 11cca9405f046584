// Column scans: the recurrence of Section 1 (Eq. 1) along T for each of J columns whose
// steps are strided in memory, for the time-major [T, N] layout (a column is an environment,
// consecutive environments are adjacent) and for F-vector eligibility traces [N, T, F] (a
// column is one feature of one row; every feature of a step shares the step's flags and so
// its coefficient beta_t, Section 3.3.5).
//
// Geometry: column j = b * C + c (batch row b, column c within it) holds step t at element
//   (j / C) * bstride + (j % C) + t * st,
// and its flags at the same element (`fcol`, time-major) or at (j / C) * fbstride + t * fst
// (one flag per step of a batch row, vector traces). The per-column row value (bootstrap) is
// element j of its array.
//
// Lanes own columns, so consecutive lanes read consecutive elements of a step (coalesced),
// and a lane's K steps are consecutive in time. A workgroup of W waves covers 64 columns and
// W*K consecutive steps (a chunk): wave w owns steps t0 + w*K .. t0 + w*K + K-1. Per lane:
//   1. load the K steps (flags first, then data, the neighbour step on the carry-source side
//      and the row value; continuation values only at truncated steps, once the flags are in);
//   2. build alpha, beta with the estimator's policy (Table 1, Section 3.2);
//   3. compose the K steps serially into one affine map;
//   4. compose the maps of the waves on the carry-source side (LDS);
//   5. take the value entering the chunk (previous chunk of the same workgroup, or the
//      published maps of other workgroups' tiles) and finish the K steps; store.
// cols_rows_kernel walks all of T in chunks (carry through LDS); cols_narrow_kernel does the
// same for narrow groups of 16 or 32 columns, whose lane groups also split time (short columns,
// a few thousand of them); cols_tiles_kernel gives each tile (kColSplitW waves, twice a walk's
// chunk) its own workgroup and carries between them with the split-row kernel's workspace
// protocol, per column: a tile publishes its 64 composed maps and composes the maps of the
// tiles on its carry-source side, nearest first, until it meets beta = 0 (an episode or row
// edge), over block aggregates when a look-back can be long. Tiles only ever wait for tiles of
// their own column block, so each block has its own draw slot: its tickets order the block's
// tiles from the carry source, and no counter is touched by every workgroup of the grid.
//
// Workspace of cols_tiles_kernel: the split layout of rlcs_kernels.h (zero-filled once), with
// one draw slot per 64-column block (at most kWsSlots blocks), records at index (offset of the
// level + block) * J + j for column j (level 0: tile of ticket t at t * J + j), and even tags
// (tag0 = 2*gen + 2, tag1 = tag0 + J * kTagMix).
#pragma once

#include "rlcs_kernels.h"

namespace rlcs {

struct ColGeom {
    int64_t J;         // columns
    int64_t C;         // columns per batch row
    int64_t st;        // elements between consecutive steps of a column
    int64_t bstride;   // elements between batch rows
    int64_t fst;       // flags between consecutive steps (flags not per column)
    int64_t fbstride;  // flags between batch rows (flags not per column)
    int fcol;          // flags laid out like the data
    // Outputs by non-temporal stores (the kernels' NT). They suit steps whose 64 columns fill
    // whole 128-byte lines; where a batch row holds fewer (vector traces of F % 32 != 0) each
    // partial line would go to memory as a whole one, and plain stores, merged in L2, write less.
    int nt_store;
};

constexpr int kColK = 8;  // steps per lane
constexpr int kColW = 4;  // waves per workgroup (time sub-spans of a chunk)
constexpr int kColL = kColK * kColW;  // steps per chunk
// Split columns: waves per workgroup of the one-tile-per-workgroup kernel, whose tiles are
// twice as long as a whole-column walk's chunks (fewer tiles to chain, more steps in flight)
constexpr int kColSplitW = 8;
constexpr int kColSplitL = kColK * kColSplitW;

// One lane's K steps of one column.
template <class Op, typename DT, int K, bool TR>
struct ColChunk {
    static constexpr bool kBack = Op::kBackward;
    static constexpr int NS = Op::kSlots;
    static constexpr int NB = Op::kNbr > 0 ? Op::kNbr : 1;
    static constexpr int kTS = TR ? Op::kTruncSlot : -1;

    float d[NS][K];
    float B[K];
    float nb[NB];
    float al[K], be[K];
    uint32_t term, trunc, edge, valid;
    int64_t t0;

    // Raw loads between issue and complete.
    uint8_t tb[K], rb[K];
    uint8_t pt, pr;
    float nraw[Op::kNbrRaw];
    float rv;
    bool have_nbr;

    // Step 1, first half. `base`: element of step 0 of the column; `fbase`, `fstep`: its flags.
    // Every load goes out unconditionally from a clamped, in-range step (the values of steps
    // past T and of inactive lanes are dropped in `complete`), so no branch waits for a load
    // and the loads of the next chunk can be in flight while this one is scanned. With
    // kBvAlways the continuation values are read here too, for every step; otherwise
    // `complete` reads them only at truncated steps.
    template <bool kBvAlways>
    __device__ __forceinline__ void issue(const Args& a, bool active, int64_t j, int64_t base,
                                          int64_t st, int64_t fbase, int64_t fstep, int64_t t0_) {
        t0 = t0_;
        const int64_t T = a.T;
        valid = 0;
        if (active) {
#pragma unroll
            for (int k = 0; k < K; ++k)
                if (t0 + k < T) valid |= 1u << k;
        }
        const uint8_t* fallback = reinterpret_cast<const uint8_t*>(a.in[0]);
#pragma unroll
        for (int k = 0; k < K; ++k) {
            const int64_t tc = min(t0 + k, T - 1);
            tb[k] = (Op::kFlags ? (a.term ? a.term : fallback) : fallback)[fbase + tc * fstep];
            rb[k] = TR ? a.trunc[fbase + tc * fstep] : uint8_t(0);
        }
#pragma unroll
        for (int s = 0; s < NS; ++s) {
#pragma unroll
            for (int k = 0; k < K; ++k) {
                const int64_t tc = min(t0 + k, T - 1);
                d[s][k] = 0.f;
                if (Op::slot_used(s, TR) && (s != kTS || kBvAlways))
                    d[s][k] = load_one<DT>(a.in[s], base + tc * st);
            }
        }
        have_nbr = false;
        pt = pr = 0;
        if constexpr (kBack) {
            if constexpr (Op::kNbr > 0) {
                Op::template nbr_load_raw<DT>(a, base + min(t0 + K, T - 1) * st, nraw);
                have_nbr = t0 + K < T;
            }
            rv = (Op::kRowValue && a.row_value) ? load_one<DT>(a.row_value, active ? j : 0) : 0.f;
        } else {
            if constexpr (Op::kNbr > 0) {
                // the step before the lane's first one, clamped into the column (a lane past
                // the column's end drops it)
                const int64_t tp = min(max(t0 - 1, int64_t(0)), T - 1);
                pt = (a.term ? a.term : fallback)[fbase + tp * fstep];
                pr = TR ? a.trunc[fbase + tp * fstep] : uint8_t(0);
            }
            rv = 0.f;
        }
    }

    // Step 1, second half: flag masks, edge, row value, neighbour; continuation values at
    // truncated steps unless `issue` read them all.
    template <bool kBvAlways>
    __device__ __forceinline__ void complete(const Args& a, int64_t base, int64_t st) {
        const int64_t T = a.T;
        term = 0;
        trunc = 0;
#pragma unroll
        for (int k = 0; k < K; ++k) {
            if (Op::kFlags && a.term && tb[k]) term |= 1u << k;
            if (TR && rb[k]) trunc |= 1u << k;
        }
        term &= valid;
        trunc &= valid;
        edge = 0;
#pragma unroll
        for (int k = 0; k < K; ++k) B[k] = 0.f;
        if (valid) {
            if (kBack) {
                if (t0 + K >= T) {  // the column's last step T-1 is among the lane's steps
                    const int ke = int(T - 1 - t0);
                    edge = 1u << ke;
#pragma unroll
                    for (int k = 0; k < K; ++k)
                        if (k == ke) B[k] = rv;
                }
            } else if (t0 == 0) {
                edge = 1u;
            }
        }
        if constexpr (kTS >= 0 && !kBvAlways) {
#pragma unroll
            for (int k = 0; k < K; ++k) {
                d[kTS][k] = 0.f;
                if (bit(trunc, k)) d[kTS][k] = load_one<DT>(a.in[kTS], base + (t0 + k) * st);
            }
        }
#pragma unroll
        for (int i = 0; i < NB; ++i) nb[i] = 0.f;
        if constexpr (kBack) {
            if (have_nbr && valid) Op::nbr_fix(a, nraw, nb);
        } else if constexpr (Op::kNbr > 0) {
            // a missing termination array was read from the data instead: its byte is dropped
            nb[0] = (t0 > 0 && ((a.term && pt) || (TR && pr))) ? 1.f : 0.f;
        }
    }

    // Step 1 without overlap: issue, then complete.
    __device__ __forceinline__ void load(const Args& a, bool active, int64_t j, int64_t base,
                                         int64_t st, int64_t fbase, int64_t fstep, int64_t t0_) {
        issue<false>(a, active, j, base, st, fbase, fstep, t0_);
        complete<false>(a, base, st);
    }

    // Steps 2-3: the lane's map (nearest-to-output step outermost).
    __device__ __forceinline__ Pair local(const Params& P) {
        Op::template build<K, TR>(P, d, term, trunc, edge, B, nb, al, be);
#pragma unroll
        for (int k = 0; k < K; ++k)
            if (!bit(valid, k)) { al[k] = 0.f; be[k] = 1.f; }
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
        return agg;
    }

    // Step 5 given X, the value entering the lane's steps from the carry-source side. Returns
    // the value of the lane's step nearest the output side.
    template <bool NT>
    __device__ __forceinline__ float finish(const Args& a, const Params& P, int64_t base, int64_t st, float X) {
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
        Op::template finish<K, TR>(P, d, term, trunc, edge, B, nb, A, X, o0, o1);
#pragma unroll
        for (int k = 0; k < K; ++k) {
            if (!bit(valid, k)) continue;
            const int64_t e = base + (t0 + k) * st;
            if constexpr (NT) {
                __builtin_nontemporal_store(o0[k], a.out0 + e);
                if (a.out1) __builtin_nontemporal_store(o1[k], a.out1 + e);
            } else {
                a.out0[e] = o0[k];
                if (a.out1) a.out1[e] = o1[k];
            }
        }
        return kBack ? A[0] : A[K - 1];
    }
};

// Two 64-column blocks share a 128-byte line of flags; the dispatcher deals workgroup b to XCD
// b mod 8, so in every run of 16 workgroups b and b+8 take blocks 2m and 2m+1 (one L2 fetches
// the line).
__device__ __forceinline__ int64_t paired_block(int64_t b, int64_t blocks) {
    const int64_t dealt = blocks / 16 * 16;
    if (b >= dealt) return b;
    return b / 16 * 16 + (b % 8) * 2 + (b / 8) % 2;
}

// Per-lane column placement.
struct ColLane {
    int64_t j, base, fbase, fstep;
    bool active;
};

__device__ __forceinline__ ColLane col_lane(const ColGeom& g, int64_t block) {
    ColLane l;
    l.j = block * kWave + (threadIdx.x & (kWave - 1));
    l.active = l.j < g.J;
    const int64_t jj = l.active ? l.j : 0;
    const int64_t b = jj / g.C, c = jj - b * g.C;
    l.base = b * g.bstride + c;
    l.fbase = g.fcol ? l.base : b * g.fbstride;
    l.fstep = g.fcol ? g.st : g.fst;
    return l;
}

// Composition of the maps of the waves on wave `wave`'s carry-source side (LDS, per lane).
template <bool kBack, int W>
__device__ __forceinline__ Pair cols_wave_in(const float (*s_a)[kWave], const float (*s_b)[kWave],
                                             int wave, int lane) {
    Pair acc = identity_pair();
    if (kBack) {
        for (int w = W - 1; w > wave; --w) acc = compose(Pair{s_a[w][lane], s_b[w][lane]}, acc);
    } else {
        for (int w = 0; w < wave; ++w) acc = compose(Pair{s_a[w][lane], s_b[w][lane]}, acc);
    }
    return acc;
}

// Whole columns per workgroup: chunks walked from the carry source, the value at the chunk's
// output-side edge carried to the next chunk through LDS. PIPE (columns of several chunks):
// the next chunk's loads are in flight while a chunk is scanned. Grid: ceil(J / 64)
// workgroups.
template <class Op, typename DT, int K, int W, bool TR, bool PIPE, bool NT = true>
__global__ void __launch_bounds__(W * kWave) cols_rows_kernel(Args a, ColGeom g) {
    constexpr bool kBack = Op::kBackward;
    constexpr int64_t L = int64_t(W) * K;
    __shared__ float s_a[W][kWave], s_b[W][kWave];
    __shared__ float s_carry[kWave];
    const int lane = threadIdx.x & (kWave - 1), wave = threadIdx.x / kWave;
    const ColLane cl = col_lane(g, paired_block(blockIdx.x, gridDim.x));
    const int64_t T = a.T;
    const int64_t P = (T + L - 1) / L;
    float carry = 0.f;
    auto t0_of = [&](int64_t i) { return (kBack ? P - 1 - i : i) * L + int64_t(wave) * K; };
    // steps 1 (second half) to 5 of chunk i, whose loads are issued; the carry moves on
    auto scan = [&](ColChunk<Op, DT, K, TR>& c) {
        c.template complete<PIPE>(a, cl.base, g.st);
        const Pair m = c.local(a.p);
        s_a[wave][lane] = m.a;
        s_b[wave][lane] = m.b;
        __syncthreads();
        const Pair win = cols_wave_in<kBack, W>(s_a, s_b, wave, lane);
        const float out_edge = c.template finish<NT>(a, a.p, cl.base, g.st, apply(win, carry));
        if (wave == (kBack ? 0 : W - 1)) s_carry[lane] = out_edge;
        __syncthreads();
        carry = s_carry[lane];
    };
    ColChunk<Op, DT, K, TR> c;
    c.template issue<PIPE>(a, cl.active, cl.j, cl.base, g.st, cl.fbase, cl.fstep, t0_of(0));
    if constexpr (PIPE) {
        // software pipeline: chunk i+1's loads (continuation values included, so that nothing
        // waits for the flags) go out before chunk i is scanned
        for (int64_t i = 0; i + 1 < P; ++i) {
            ColChunk<Op, DT, K, TR> nxt;
            nxt.template issue<true>(a, cl.active, cl.j, cl.base, g.st, cl.fbase, cl.fstep, t0_of(i + 1));
            __builtin_amdgcn_sched_barrier(0);  // keep those loads ahead of this chunk's first wait
            scan(c);
            c = nxt;
        }
        scan(c);
    } else {
        for (int64_t i = 0;; ++i) {
            scan(c);
            if (i + 1 == P) break;
            c.template issue<false>(a, cl.active, cl.j, cl.base, g.st, cl.fbase, cl.fstep, t0_of(i + 1));
        }
    }
}

// Narrow column groups, whole columns per workgroup, no workspace: a workgroup serves
// kNarrowCols(DT) columns (64 bytes of a step: 16 float32 or 32 bfloat16 columns), so that a
// few thousand columns already give every CU a workgroup without splitting columns in time.
// Lane l of a wave owns column l mod C and the (l / C)-th of the wave's 64/C lane groups, which
// take consecutive time spans of K steps, as the W waves of the workgroup do: one chunk is
// (64/C)*W*K steps. Per chunk, a lane's K steps compose serially, the lane groups of a wave
// scan by shuffles, the waves compose through LDS, and the carry passes to the next chunk
// through LDS. A 128-byte line of data spans two column groups and a line of flags eight
// (float32; four for bfloat16). The dispatcher deals workgroup b to XCD b mod 8, so in every run
// of 64 workgroups the eight of XCD x take groups 8x .. 8x+7: each line is fetched by one L2.
// Grid: one workgroup per column group.
template <typename DT>
constexpr int narrow_cols() { return 64 / int(sizeof(DT)); }

__device__ __forceinline__ int64_t narrow_group(int64_t b, int64_t groups) {
    const int64_t dealt = groups / 64 * 64;
    if (b >= dealt) return b;
    return b / 64 * 64 + (b % 8) * 8 + (b / 8) % 8;
}

template <class Op, typename DT, int K, int W, bool TR, bool PIPE, bool NT = true>
__global__ void __launch_bounds__(W * kWave) cols_narrow_kernel(Args a, ColGeom g, int64_t groups) {
    constexpr bool kBack = Op::kBackward;
    constexpr int C = narrow_cols<DT>();
    constexpr int G = kWave / C;  // lane groups per wave
    constexpr int64_t L = int64_t(G) * W * K;
    __shared__ float s_a[W][C], s_b[W][C];
    __shared__ float s_carry[C];
    const int lane = threadIdx.x & (kWave - 1), wave = threadIdx.x / kWave;
    const int col = lane % C, grp = lane / C;
    ColLane cl;
    cl.j = narrow_group(blockIdx.x, groups) * C + col;
    cl.active = cl.j < g.J;
    {
        const int64_t jj = cl.active ? cl.j : 0;
        const int64_t b = jj / g.C, c = jj - b * g.C;
        cl.base = b * g.bstride + c;
        cl.fbase = g.fcol ? cl.base : b * g.fbstride;
        cl.fstep = g.fcol ? g.st : g.fst;
    }
    const int64_t T = a.T;
    const int64_t P = (T + L - 1) / L;
    const int span = wave * G + grp;  // the lane's K steps within the chunk, in time order
    float carry = 0.f;
    auto t0_of = [&](int64_t i) { return (kBack ? P - 1 - i : i) * L + int64_t(span) * K; };
    auto scan = [&](ColChunk<Op, DT, K, TR>& c) {
        c.template complete<PIPE>(a, cl.base, g.st);
        const Pair m = c.local(a.p);
        // lane groups of the wave: inclusive scan from the carry-source side, then the
        // composition of the groups on this group's carry-source side
        Pair incl = m;
#pragma unroll
        for (int d = 1; d < G; d <<= 1) {
            const int src = kBack ? lane + d * C : lane - d * C;
            const Pair o{__shfl(incl.a, src), __shfl(incl.b, src)};
            if (kBack ? (grp + d < G) : (grp >= d)) incl = compose(incl, o);
        }
        const int nsrc = kBack ? lane + C : lane - C;
        const Pair nxt{__shfl(incl.a, nsrc), __shfl(incl.b, nsrc)};
        const Pair grp_in = (kBack ? (grp + 1 < G) : (grp > 0)) ? nxt : identity_pair();
        if (grp == (kBack ? 0 : G - 1)) {  // this lane's incl is the whole wave's map
            s_a[wave][col] = incl.a;
            s_b[wave][col] = incl.b;
        }
        __syncthreads();
        Pair win = identity_pair();
        if (kBack) {
            for (int w = W - 1; w > wave; --w) win = compose(Pair{s_a[w][col], s_b[w][col]}, win);
        } else {
            for (int w = 0; w < wave; ++w) win = compose(Pair{s_a[w][col], s_b[w][col]}, win);
        }
        const float X = apply(grp_in, apply(win, carry));
        const float out_edge = c.template finish<NT>(a, a.p, cl.base, g.st, X);
        if (span == (kBack ? 0 : G * W - 1)) s_carry[col] = out_edge;
        __syncthreads();
        carry = s_carry[col];
    };
    ColChunk<Op, DT, K, TR> c;
    c.template issue<PIPE>(a, cl.active, cl.j, cl.base, g.st, cl.fbase, cl.fstep, t0_of(0));
    if constexpr (PIPE) {
        for (int64_t i = 0; i + 1 < P; ++i) {
            ColChunk<Op, DT, K, TR> nxt;
            nxt.template issue<true>(a, cl.active, cl.j, cl.base, g.st, cl.fbase, cl.fstep, t0_of(i + 1));
            __builtin_amdgcn_sched_barrier(0);  // keep those loads ahead of this chunk's first wait
            scan(c);
            c = nxt;
        }
        scan(c);
    } else {
        for (int64_t i = 0;; ++i) {
            scan(c);
            if (i + 1 == P) break;
            c.template issue<false>(a, cl.active, cl.j, cl.base, g.st, cl.fbase, cl.fstep, t0_of(i + 1));
        }
    }
}

// Look-back over block aggregates, in ticket space (ticket 0 holds the column's carry-source
// edge; a tile's carry comes from the tiles of lower tickets). Level-l block q of a column is
// the tiles of tickets [q * 2^l, (q + 1) * 2^l); its map composes the maps of its two halves,
// the upper half outermost, and is published by the block's last ticket, which finishes the
// levels its ticket t closes (2^l divides t + 1) one after the other, each waiting for the lower
// half's map. The value entering tile t composes, nearest first, the blocks of a fixed
// decomposition of [0, t): from y = t down, a block [y - 2^l, y) with l the lesser of the
// number of trailing zero bits of y and (steps taken - kColLiftAfter), so the first steps read
// single tiles and later ones doubling blocks: O(log t) reads down to the edge. It stops at the
// first block with beta = 0 (an episode edge; ticket 0 always holds one). The decomposition
// depends only on t and every block composes in a fixed order, so results are bitwise
// reproducible; a column without flags and gamma*lambda = 1 no longer reads all t maps.
// Building the blocks makes some workgroups wait for chains of them, so the host asks for them
// (`lift`) only when a look-back can be long: when the product of the betas of a run of tiles
// cannot underflow to 0 within a few dozen tiles. Otherwise every block read is a single tile.
// Records of level l start at block sum over l' < l of (P >> l'); a record is two 64-bit words
// per column at index (offset + q) * J + j.
constexpr int kColLookAhead = 4;
constexpr int kColLiftAfter = 3;

__device__ __forceinline__ int64_t col_level_offset(int64_t P, int l) {
    int64_t off = 0;
    for (int k = 0; k < l; ++k) off += P >> k;
    return off;
}

__device__ __forceinline__ Pair col_wait_record(const uint64_t* r, uint32_t tag0, uint32_t tag1,
                                                uint64_t w0, uint64_t w1, WsHeader* hdr, bool& ok) {
    uint32_t polls = 0;
    while (uint32_t(w0 >> 32) != tag0 || uint32_t(w1 >> 32) != tag1) {
        if (++polls > kMaxPolls) {
            st_relaxed(&hdr->error, 1u);
            ok = false;
            return Pair{__builtin_nanf(""), 0.f};
        }
        __builtin_amdgcn_s_sleep(1);
        w0 = ld_relaxed(r);
        w1 = ld_relaxed(r + 1);
    }
    return Pair{__uint_as_float(uint32_t(w0)), __uint_as_float(uint32_t(w1))};
}

// Value entering the tile of ticket t (t > 0) in column j. Bounded polls: on exhaustion the
// error flag is set and NaN returned.
template <bool LIFT>
__device__ float cols_gather(const uint64_t* rec, int64_t t, int64_t P, int64_t J, int64_t j,
                             uint32_t tag0, uint32_t tag1, WsHeader* hdr) {
    Pair acc = identity_pair();
    if constexpr (!LIFT) {
        // single tiles only: tickets t-1, t-2, ..., kColLookAhead per round
        for (int64_t d = 1;; d += kColLookAhead) {
            uint64_t w0[kColLookAhead], w1[kColLookAhead];
#pragma unroll
            for (int i = 0; i < kColLookAhead; ++i) {
                const int64_t q = t - d - i;
                w0[i] = w1[i] = 0;
                if (q >= 0) {
                    w0[i] = ld_relaxed(rec + 2 * (q * J + j));
                    w1[i] = ld_relaxed(rec + 2 * (q * J + j) + 1);
                }
            }
#pragma unroll
            for (int i = 0; i < kColLookAhead; ++i) {
                const int64_t q = t - d - i;
                if (q < 0) return acc.a;  // past the edge tile (not reached: its beta is 0)
                bool ok = true;
                const Pair m = col_wait_record(rec + 2 * (q * J + j), tag0, tag1, w0[i], w1[i], hdr, ok);
                if (!ok) return __builtin_nanf("");
                acc = compose(acc, m);
                if (m.b == 0.f) return acc.a;
            }
        }
    }
    int64_t y = t;
    int step = 0;
    while (y > 0) {
        // the next kColLookAhead blocks of the decomposition, read together
        const uint64_t* r[kColLookAhead];
        uint64_t w0[kColLookAhead], w1[kColLookAhead];
        int n = 0;
        int64_t yy = y;
#pragma unroll
        for (int k = 0; k < kColLookAhead; ++k) {
            r[k] = nullptr;
            w0[k] = w1[k] = 0;
            if (yy > 0) {
                const int lim = max(step + k - kColLiftAfter, 0);
                const int l = min(int(__builtin_ctzll(uint64_t(yy))), lim);
                const int64_t q = (yy >> l) - 1;
                r[k] = rec + 2 * ((col_level_offset(P, l) + q) * J + j);
                w0[k] = ld_relaxed(r[k]);
                w1[k] = ld_relaxed(r[k] + 1);
                yy -= int64_t(1) << l;
                n = k + 1;
            }
        }
#pragma unroll
        for (int k = 0; k < kColLookAhead; ++k) {
            if (k >= n) break;
            bool ok = true;
            const Pair m = col_wait_record(r[k], tag0, tag1, w0[k], w1[k], hdr, ok);
            if (!ok) return __builtin_nanf("");
            acc = compose(acc, m);
            if (m.b == 0.f) return acc.a;
        }
        y = yy;
        step += n;
    }
    return acc.a;  // not reached: ticket 0's map has beta = 0
}

// Publishes the level-l maps that ticket t closes (block [t + 1 - 2^l, t + 1) for every l with
// 2^l dividing t + 1), starting from `m`, the tile's own map; each waits for the map of the
// block's lower half.
__device__ void cols_publish_levels(uint64_t* rec, int64_t t, int64_t P, int64_t J, int64_t j,
                                    Pair m, uint32_t tag0, uint32_t tag1, WsHeader* hdr) {
    int64_t off_prev = 0;  // offset of level l - 1
    for (int l = 1; l < 63 && ((t + 1) & ((int64_t(1) << l) - 1)) == 0; ++l) {
        const int64_t q = ((t + 1) >> l) - 1;           // this block at level l
        const int64_t lower = 2 * q;                     // its lower half at level l - 1
        const uint64_t* r = rec + 2 * ((off_prev + lower) * J + j);
        bool ok = true;
        const Pair h = col_wait_record(r, tag0, tag1, ld_relaxed(r), ld_relaxed(r + 1), hdr, ok);
        if (!ok) return;
        m = compose(m, h);
        const int64_t off = off_prev + (P >> (l - 1));
        uint64_t* w = rec + 2 * ((off + q) * J + j);
        st_relaxed(w, uint64_t(tag0) << 32 | __float_as_uint(m.a));
        st_relaxed(w + 1, uint64_t(tag1) << 32 | __float_as_uint(m.b));
        off_prev = off;
    }
}

// The n of a column call's tag1: the column count and which split kernel cut the columns into
// blocks (0: 64-column blocks; 1, 2: narrow groups of 16 float32 or 32 bfloat16 columns), since a
// column's draw slot depends on both. Distinct for every (J, kind) with J < 2^30.
__device__ __forceinline__ uint32_t col_tag_n(int64_t J, int kind) { return uint32_t(J) * 4u + uint32_t(kind); }

// One chunk per workgroup. Workgroup g serves column block g mod num_blocks; its ticket among
// that block's P workgroups orders the block's tiles from the carry source, so a tile only waits
// for tiles of its block that drew earlier tickets. LIFT: publish and read block aggregates.
// Grid: num_blocks * P workgroups.
template <class Op, typename DT, int K, int W, bool TR, bool LIFT, bool NT = true>
__global__ void __launch_bounds__(W * kWave) cols_tiles_kernel(Args a, ColGeom g, int64_t num_blocks) {
    constexpr bool kBack = Op::kBackward;
    constexpr int64_t L = int64_t(W) * K;
    static_assert(W >= 2, "wave 1 publishes the block aggregates while wave 0 looks back");
    __shared__ float s_a[W][kWave], s_b[W][kWave];
    __shared__ float s_carry[kWave];
    __shared__ uint32_t s_ticket, s_tag;
    WsHeader* hdr = reinterpret_cast<WsHeader*>(a.ws);
    uint64_t* rec = reinterpret_cast<uint64_t*>(reinterpret_cast<char*>(a.ws) + kWsRecordsOffset);
    const int lane = threadIdx.x & (kWave - 1), wave = threadIdx.x / kWave;
    const int64_t T = a.T;
    const int64_t P = (T + L - 1) / L;
    const int64_t block = num_blocks % 8 == 0 ? paired_block(int64_t(blockIdx.x) % num_blocks, num_blocks)
                                              : int64_t(blockIdx.x) % num_blocks;

    if (threadIdx.x == 0) {
        uint32_t gen;
        s_ticket = draw_ticket(draw_word(a.ws, block), P, gen);
        s_tag = 2u * gen + 2u;
    }
    __syncthreads();
    const uint32_t tag0 = s_tag;
    const uint32_t tag1 = tag0 + col_tag_n(g.J, 0) * kTagMix;
    const int64_t ticket = s_ticket;
    if (wave == 0) advance_idle_slots(a.ws, num_blocks, (tag0 - 2u) / 2u, lane);
    if (ticket >= P) {
        // Only possible if the workspace was not zero-filled before first use.
        if (threadIdx.x == 0) st_relaxed(&hdr->error, 1u);
        return;
    }
    const int64_t p = kBack ? P - 1 - ticket : ticket;
    const ColLane cl = col_lane(g, block);

    ColChunk<Op, DT, K, TR> c;
    c.load(a, cl.active, cl.j, cl.base, g.st, cl.fbase, cl.fstep, p * L + int64_t(wave) * K);
    const Pair m = c.local(a.p);
    s_a[wave][lane] = m.a;
    s_b[wave][lane] = m.b;
    __syncthreads();
    const Pair win = cols_wave_in<kBack, W>(s_a, s_b, wave, lane);
    // In ticket space: a tile is read by higher tickets unless it is the last one, and needs a
    // carry unless it holds the carry-source edge (ticket 0).
    const bool publish = ticket < P - 1;
    const bool need = ticket > 0;
    if ((wave == 0 || (wave == 1 && LIFT)) && publish && cl.active) {
        // the whole tile's map of this column
        Pair tm = identity_pair();
        if (kBack) {
            for (int w = W - 1; w >= 0; --w) tm = compose(Pair{s_a[w][lane], s_b[w][lane]}, tm);
        } else {
            for (int w = 0; w < W; ++w) tm = compose(Pair{s_a[w][lane], s_b[w][lane]}, tm);
        }
        if (wave == 0) {
            st_relaxed(rec + 2 * (ticket * g.J + cl.j), uint64_t(tag0) << 32 | __float_as_uint(tm.a));
            st_relaxed(rec + 2 * (ticket * g.J + cl.j) + 1, uint64_t(tag1) << 32 | __float_as_uint(tm.b));
        } else {
            cols_publish_levels(rec, ticket, P, g.J, cl.j, tm, tag0, tag1, hdr);
        }
    }
    if (wave == 0)
        s_carry[lane] = (need && cl.active) ? cols_gather<LIFT>(rec, ticket, P, g.J, cl.j, tag0, tag1, hdr) : 0.f;
    __syncthreads();
    c.template finish<NT>(a, a.p, cl.base, g.st, apply(win, s_carry[lane]));
}

// Split tiles over narrow column groups (16 float32 or 32 bfloat16 columns per block, the lane
// layout of cols_narrow_kernel): up to four (two) times the workgroups of 64-column tiles for
// calls of few, long columns, with the draw slots, records and look-back of cols_tiles_kernel
// (per block of C columns); tiles of G * W * K steps. Grid: num_blocks * P workgroups.
// With `dealt` set (the dispatcher sets it only when the whole grid is resident at once and P
// is a multiple of 8), the tiles are dealt statically instead of drawn: workgroup b runs on XCD
// x = b mod 8, and its r = b / 8 serves block r mod num_blocks at tile x * P/8 + r / num_blocks,
// so each XCD takes a contiguous eighth of the tiles of every block. The blocks of one tile,
// which share lines of data (two float32 blocks) and of flags (all the blocks of a flag row),
// then run on one XCD, and each line is fetched by one L2; drawn in arrival order, they run on
// different XCDs. A static order needs every workgroup resident, as a tile waits on the one
// before it.
template <class Op, typename DT, int K, int W, bool TR, bool LIFT, bool NT = true>
__global__ void __launch_bounds__(W * kWave) cols_narrow_tiles_kernel(Args a, ColGeom g,
                                                                      int64_t num_blocks, int dealt) {
    constexpr bool kBack = Op::kBackward;
    constexpr int C = narrow_cols<DT>();
    constexpr int G = kWave / C;
    constexpr int64_t L = int64_t(G) * W * K;
    static_assert(W >= 2, "wave 1 publishes the block aggregates while wave 0 looks back");
    __shared__ float s_a[W][C], s_b[W][C];
    __shared__ float s_carry[C];
    __shared__ uint32_t s_ticket, s_tag;
    WsHeader* hdr = reinterpret_cast<WsHeader*>(a.ws);
    uint64_t* rec = reinterpret_cast<uint64_t*>(reinterpret_cast<char*>(a.ws) + kWsRecordsOffset);
    const int lane = threadIdx.x & (kWave - 1), wave = threadIdx.x / kWave;
    const int col = lane % C, grp = lane / C;
    const int64_t T = a.T;
    const int64_t P = (T + L - 1) / L;
    const int64_t r = int64_t(blockIdx.x) / 8;
    const int64_t block = dealt ? r % num_blocks : int64_t(blockIdx.x) % num_blocks;

    if (threadIdx.x == 0) {
        uint32_t gen;  // dealt tiles draw too: the P-th draw moves the slot to the next generation
        s_ticket = draw_ticket(draw_word(a.ws, block), P, gen);
        s_tag = 2u * gen + 2u;
    }
    __syncthreads();
    const uint32_t tag0 = s_tag;
    const uint32_t tag1 = tag0 + col_tag_n(g.J, sizeof(DT) == 4 ? 1 : 2) * kTagMix;
    if (wave == 0) advance_idle_slots(a.ws, num_blocks, (tag0 - 2u) / 2u, lane);
    if (s_ticket >= P) {
        // Only possible if the workspace was not zero-filled before first use.
        if (threadIdx.x == 0) st_relaxed(&hdr->error, 1u);
        return;
    }
    const int64_t ticket = dealt ? int64_t(blockIdx.x % 8) * (P / 8) + r / num_blocks : int64_t(s_ticket);
    const int64_t p = kBack ? P - 1 - ticket : ticket;
    ColLane cl;
    cl.j = block * C + col;
    cl.active = cl.j < g.J;
    {
        const int64_t jj = cl.active ? cl.j : 0;
        const int64_t b = jj / g.C, c = jj - b * g.C;
        cl.base = b * g.bstride + c;
        cl.fbase = g.fcol ? cl.base : b * g.fbstride;
        cl.fstep = g.fcol ? g.st : g.fst;
    }
    const int span = wave * G + grp;  // the lane's K steps within the tile, in time order

    ColChunk<Op, DT, K, TR> c;
    c.load(a, cl.active, cl.j, cl.base, g.st, cl.fbase, cl.fstep, p * L + int64_t(span) * K);
    const Pair m = c.local(a.p);
    // lane groups of the wave (shuffles), then the waves (LDS), as in cols_narrow_kernel
    Pair incl = m;
#pragma unroll
    for (int d = 1; d < G; d <<= 1) {
        const int src = kBack ? lane + d * C : lane - d * C;
        const Pair o{__shfl(incl.a, src), __shfl(incl.b, src)};
        if (kBack ? (grp + d < G) : (grp >= d)) incl = compose(incl, o);
    }
    const int nsrc = kBack ? lane + C : lane - C;
    const Pair nxt{__shfl(incl.a, nsrc), __shfl(incl.b, nsrc)};
    const Pair grp_in = (kBack ? (grp + 1 < G) : (grp > 0)) ? nxt : identity_pair();
    if (grp == (kBack ? 0 : G - 1)) {
        s_a[wave][col] = incl.a;
        s_b[wave][col] = incl.b;
    }
    __syncthreads();
    Pair win = identity_pair();
    if (kBack) {
        for (int w = W - 1; w > wave; --w) win = compose(Pair{s_a[w][col], s_b[w][col]}, win);
    } else {
        for (int w = 0; w < wave; ++w) win = compose(Pair{s_a[w][col], s_b[w][col]}, win);
    }
    const bool publish = ticket < P - 1;
    const bool need = ticket > 0;
    if (grp == 0 && (wave == 0 || (wave == 1 && LIFT)) && publish && cl.active) {
        // the whole tile's map of this column
        Pair tm = identity_pair();
        if (kBack) {
            for (int w = W - 1; w >= 0; --w) tm = compose(Pair{s_a[w][col], s_b[w][col]}, tm);
        } else {
            for (int w = 0; w < W; ++w) tm = compose(Pair{s_a[w][col], s_b[w][col]}, tm);
        }
        if (wave == 0) {
            st_relaxed(rec + 2 * (ticket * g.J + cl.j), uint64_t(tag0) << 32 | __float_as_uint(tm.a));
            st_relaxed(rec + 2 * (ticket * g.J + cl.j) + 1, uint64_t(tag1) << 32 | __float_as_uint(tm.b));
        } else {
            cols_publish_levels(rec, ticket, P, g.J, cl.j, tm, tag0, tag1, hdr);
        }
    }
    if (wave == 0 && grp == 0)
        s_carry[col] = (need && cl.active) ? cols_gather<LIFT>(rec, ticket, P, g.J, cl.j, tag0, tag1, hdr) : 0.f;
    __syncthreads();
    c.template finish<NT>(a, a.p, cl.base, g.st, apply(grp_in, apply(win, s_carry[col])));
}

}  // namespace rlcs
