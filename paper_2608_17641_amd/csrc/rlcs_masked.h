// GAE with observation-skip masking (the planned extension of Section 9.3: the recurrence is
// carried across masked tokens, beta_t = 1) and optional whitening of the advantages.
//
// A masked step (an observation token) passes on both the running advantage A and the value W
// that the preceding unmasked step sees as its successor: the value of the next unmasked step.
// The pair (A, W) therefore obeys one backward recurrence whose per-step map is affine with an
// upper-triangular linear part,
//   (A, W) at t  =  [[p, q], [0, s]] (A, W) at t+1  +  (ca, cw):
//   unmasked, continuing:  A = r - V + gamma W' + gamma lambda A',   W = V;
//   unmasked, cut:         A = r - V + gamma * (0 | bv | boot),       W = V;
//   masked, continuing:    A = A', W = W';
//   masked, cut:           A = 0,  W = (0 | bv | boot);
// where a cut is a termination (successor 0), a truncation (its continuation bv_t) or the row's
// last step (the bootstrap). These maps compose associatively like the pairs of Eq. 2, so one
// segmented scan over the flat [N*T] array evaluates the recurrence: each lane composes its K
// steps, a DPP wave scan composes lanes, LDS composes waves and carries chunks.
//
// Whitening: the scan kernel also reduces the advantages of the unmasked steps of each
// workgroup to fp64 sums (count, sum, sum of squares) and stores them as the workgroup's
// partial. A second kernel rewrites the advantages: each of its workgroups first adds up all
// partials itself, in one fixed order, so every workgroup derives the same mean and
// 1/sqrt(var + eps) (var the unbiased variance) and results are reproducible bit for bit.
// The kernel boundary orders the partials before their readers, so no atomics or fences are
// needed. With more than kDirectPartials partials a small kernel in between first adds them
// in blocks of kDirectPartials. fp64 sums of fp32 advantages lose accuracy in the variance only
// when |mean| / std approaches 1e6, far past what fp32 advantages resolve anyway.
#pragma once

#include "rlcs_kernels.h"

namespace rlcs {

// (A, W) -> (p A + q W + ca, s W + cw)
struct Tri {
    float p, q, s, ca, cw;
};
struct AW {
    float A, W;
};

__device__ __forceinline__ Tri identity_tri() { return Tri{1.f, 0.f, 1.f, 0.f, 0.f}; }

__device__ __forceinline__ Tri compose(const Tri& o, const Tri& i) {
    return Tri{o.p * i.p, fmaf(o.p, i.q, o.q * i.s), o.s * i.s,
               fmaf(o.p, i.ca, fmaf(o.q, i.cw, o.ca)), fmaf(o.s, i.cw, o.cw)};
}

__device__ __forceinline__ AW apply(const Tri& m, AW x) {
    return AW{fmaf(m.p, x.A, fmaf(m.q, x.W, m.ca)), fmaf(m.s, x.W, m.cw)};
}

__device__ __forceinline__ float readlane_f(float v, int lane) {
    return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), lane));
}

__device__ __forceinline__ Tri read_lane(const Tri& v, int lane) {
    return Tri{readlane_f(v.p, lane), readlane_f(v.q, lane), readlane_f(v.s, lane),
               readlane_f(v.ca, lane), readlane_f(v.cw, lane)};
}

// One Kogge-Stone step on triangular maps with DPP-modified VALU operations, as for pairs
// (wave_scan_inclusive in the device header): a lane whose DPP source exists composes its map
// (outer) with the source's map (inner); the others are not written and keep theirs. Every
// component of the source is read before the source lane overwrites it, so q and ca are first
// copied: q' = q s_src + p q_src, ca' = ca + q cw_src + p ca_src, cw' = cw + s cw_src,
// s' = s s_src, p' = p p_src, in that order.
#define RLCS_TRI_DPP_STEP(v, CTRL)                                                            \
    {                                                                                         \
        float tq = v.q, tca = v.ca;                                                           \
        asm volatile("s_nop 1\n\tv_mul_f32_dpp %1, %2, %1 " CTRL " bank_mask:0xf\n\t"         \
                     "s_nop 1\n\tv_fmac_f32_dpp %1, %5, %0 " CTRL " bank_mask:0xf\n\t"        \
                     "s_nop 1\n\tv_fmac_f32_dpp %3, %4, %5 " CTRL " bank_mask:0xf\n\t"        \
                     "s_nop 1\n\tv_fmac_f32_dpp %3, %6, %0 " CTRL " bank_mask:0xf\n\t"        \
                     "s_nop 1\n\tv_fmac_f32_dpp %4, %4, %2 " CTRL " bank_mask:0xf\n\t"        \
                     "s_nop 1\n\tv_mul_f32_dpp %2, %2, %2 " CTRL " bank_mask:0xf\n\t"         \
                     "s_nop 1\n\tv_mul_f32_dpp %0, %0, %0 " CTRL " bank_mask:0xf"               \
                     : "+v"(v.p), "+v"(v.q), "+v"(v.s), "+v"(v.ca), "+v"(v.cw), "+v"(tq), "+v"(tca)); \
    }

// Inclusive prefix scan of per-lane maps over the 64 lanes, as wave_scan_inclusive for pairs:
// four row shifts, then the row broadcasts of lanes 15 and 31.
__device__ __forceinline__ Tri wave_scan_inclusive(Tri v, int lane) {
    (void)lane;
    RLCS_TRI_DPP_STEP(v, "row_shr:1 row_mask:0xf")
    RLCS_TRI_DPP_STEP(v, "row_shr:2 row_mask:0xf")
    RLCS_TRI_DPP_STEP(v, "row_shr:4 row_mask:0xf")
    RLCS_TRI_DPP_STEP(v, "row_shr:8 row_mask:0xf")
    RLCS_TRI_DPP_STEP(v, "row_bcast:15 row_mask:0xa")
    RLCS_TRI_DPP_STEP(v, "row_bcast:31 row_mask:0xc")
    return v;
}
#undef RLCS_TRI_DPP_STEP

// Value of lane l-1 (lane 0 receives `fill`).
__device__ __forceinline__ AW shift_up1(AW v, AW fill) {
    return AW{shift_up1(v.A, fill.A), shift_up1(v.W, fill.W)};
}

// fp64 sums of the advantages of the unmasked steps of one workgroup (or of a block of
// partials): count, sum, sum of squares.
struct alignas(32) Moments {
    double n, s1, s2, pad;
};

struct MaskedArgs {
    Args a;              // in[0] r, in[1] v, in[2] bv; term, trunc; row_value = boot;
                         // out0 adv, out1 ret (optional)
    const uint8_t* mask; // [N, T], nonzero = the step takes part; null = every step does
    // whitening only (workspace): one partial per workgroup
    Moments* partials;
};

constexpr int kDirectPartials = 4096;  // partials one normalize workgroup adds up itself

// Map of one step.
__device__ __forceinline__ Tri masked_gae_step(const Params& P, bool in, bool te, bool tr, bool ed,
                                               float r, float v, float bv, float B) {
    const bool cut = te || tr || ed;
    const float s_cut = te ? 0.f : (tr ? bv : B);
    if (in) {
        const float rv = r - v;
        return cut ? Tri{0.f, 0.f, 0.f, fmaf(P.gamma, s_cut, rv), v}
                   : Tri{P.gamma * P.lambda, P.gamma, 0.f, rv, v};
    }
    return cut ? Tri{0.f, 0.f, 0.f, 0.f, s_cut} : identity_tri();
}

// One lane's K consecutive steps of a chunk (lane l owns the (63-l)-th group of its wave's
// span: the carry flows from lane l-1 to lane l).
template <typename DT, int K, bool TR, bool HM>
struct MaskedChunk {
    static constexpr uint32_t kAll = (1u << K) - 1u;
    static constexpr int kWords = K * int(sizeof(DT)) / 4;
    float r[K], v[K], bv[K], B[K];
    uint32_t mk, term, trunc, edge, valid;
    Tri m[K];
    Tri incl;
    int64_t p0;

    // Vector loads of the lane's K steps (16-byte aligned data, T >= K, all K steps inside the
    // array; `base` a row start at or before p0), every one issued before the first use; at most
    // one row edge. `in_range` selects the steps that are the lane's: all, or those of a ragged
    // end of the workgroup's range.
    __device__ __forceinline__ void load_full(const MaskedArgs& ma, const RowBase& base,
                                              uint32_t in_range) {
        const Args& a = ma.a;
        valid = in_range;
        const uint8_t* fallback = reinterpret_cast<const uint8_t*>(a.in[0]);
        uint32_t tw[(K + 3) / 4], rw[(K + 3) / 4], mw[(K + 3) / 4];
        if (TR) load_flag_words<K>(a.trunc, p0, rw);
        load_flag_words<K>(a.term ? a.term : fallback, p0, tw);
        if (HM) load_flag_words<K>(ma.mask, p0, mw);
        uint32_t wr[kWords], wv[kWords], wb[kWords];
        load_words<DT, K>(a.in[0], p0, wr);
        load_words<DT, K>(a.in[1], p0, wv);
        int64_t row, t;
        row_and_step(base, p0, a.T, a.inv_T, row, t);
        const int ke = (t + K - 1 >= a.T - 1) ? int(a.T - 1 - t) : -1;
        const float rv_raw = load_one<DT>(a.row_value ? a.row_value : a.in[0], min(row, a.N - 1));
        trunc = TR ? flag_mask<K>(rw) : 0u;
        if (TR && trunc) load_words<DT, K>(a.in[2], p0, wb);
        else {
#pragma unroll
            for (int i = 0; i < kWords; ++i) wb[i] = 0u;
        }
        unpack_words<DT, K>(wr, r);
        unpack_words<DT, K>(wv, v);
        unpack_words<DT, K>(wb, bv);
        term = a.term ? flag_mask<K>(tw) : 0u;
        mk = HM ? flag_mask<K>(mw) : kAll;
        edge = ke >= 0 ? (1u << ke) : 0u;
        const float rv = a.row_value ? rv_raw : 0.f;
#pragma unroll
        for (int k = 0; k < K; ++k) B[k] = (k == ke) ? rv : 0.f;
    }

    // Steps of a chunk with steps outside [lo, hi): element-wise, masked.
    __device__ __forceinline__ void load_masked(const MaskedArgs& ma, const RowBase& base,
                                                int64_t lo, int64_t hi) {
        const Args& a = ma.a;
        valid = 0;
#pragma unroll
        for (int k = 0; k < K; ++k)
            if (p0 + k >= lo && p0 + k < hi) valid |= 1u << k;
        edge = 0;
#pragma unroll
        for (int k = 0; k < K; ++k) B[k] = 0.f;
        if (valid) {
            const int64_t first = p0 + __builtin_ctz(valid);
            int64_t row, t;
            row_and_step(base, first, a.T, a.inv_T, row, t);
#pragma unroll
            for (int k = 0; k < K; ++k) {
                if (p0 + k < first || !bit(valid, k)) continue;
                if (t == a.T - 1) {
                    edge |= 1u << k;
                    if (a.row_value) B[k] = load_one<DT>(a.row_value, row);
                }
                if (++t == a.T) { t = 0; ++row; }
            }
        }
        term = a.term ? load_flags_masked<K>(a.term, p0, valid) : 0u;
        trunc = TR ? load_flags_masked<K>(a.trunc, p0, valid) : 0u;
        mk = HM ? load_flags_masked<K>(ma.mask, p0, valid) : valid;
        load_k<DT, K>(a.in[0], p0, valid, false, r);
        load_k<DT, K>(a.in[1], p0, valid, false, v);
        load_k<DT, K>(a.in[2], p0, valid & trunc, false, bv);
    }

    // The lane's composed map (step 0 outermost) and its inclusive wave scan.
    __device__ __forceinline__ Tri local(const Params& P, int lane) {
#pragma unroll
        for (int k = 0; k < K; ++k)
            m[k] = bit(valid, k) ? masked_gae_step(P, bit(mk, k), bit(term, k), TR && bit(trunc, k),
                                                   bit(edge, k), r[k], v[k], bv[k], B[k])
                                 : identity_tri();
        Tri agg = m[K - 1];
#pragma unroll
        for (int k = K - 2; k >= 0; --k) agg = compose(m[k], agg);
        incl = wave_scan_inclusive(agg, lane);
        return incl;
    }

    // Outputs given Xw, the state entering the wave's span; returns the state at the lane's
    // first step. Accumulates the advantages that take part into (n, sum, sumsq). `full`: the
    // lane's steps are vector-aligned (stored as vectors when all of them are the lane's).
    float adv[K];  // the lane's advantages (kept for the fused whitening)
    // K = 8: the wave's LDS slot for whole-line stores. A wave whose lanes all store whole
    // vectors holds 512 consecutive outputs (lane l the group 63 - l of them).
    f32x4* oslot = nullptr;

    // Stores the lane's K outputs `v` to `out`: whole lines through the wave's slot when every
    // lane of the wave stores whole vectors (K = 8), else per lane.
    __device__ __forceinline__ void store(float* out, bool vstore, const float (&v)[K]) {
        if constexpr (K == 8) {
            if (__all(vstore)) {
                const int lane = threadIdx.x & (kWave - 1);
                const int g = kWave - 1 - lane;
                const int64_t base = p0 - int64_t(g) * K;
                store8_lines(out, base, base + kWave * K, g, lane, v, oslot);
                return;
            }
        }
        store_k<K>(out, p0, valid, vstore, v);
    }

    template <bool STATS, bool STORE_ADV = true>
    __device__ __forceinline__ AW finish(const Args& a, AW Xw, bool full, double& n, double& s1,
                                         double& s2) {
        AW x = shift_up1(apply(incl, Xw), Xw);
        float ret[K];
#pragma unroll
        for (int k = K - 1; k >= 0; --k) {
            x = apply(m[k], x);
            adv[k] = x.A;
            ret[k] = x.A + v[k];
            if (STATS && bit(valid, k) && bit(mk, k)) {
                const double d = double(x.A);
                n += 1.0;
                s1 += d;
                s2 = fma(d, d, s2);
            }
        }
        const bool vstore = full && valid == kAll;
        if (STORE_ADV) store(a.out0, vstore, adv);
        if (a.out1) store(a.out1, vstore, ret);
        return x;
    }
};

// Sum over the 64 lanes in fp64, the same value in every lane, in one fixed order: a DPP
// prefix sum inside each row of 16 lanes (both 32-bit halves moved by row shifts, zeros shifted
// in), then the four row totals read as scalars. Against a shuffle butterfly (12 LDS-speed
// permutes per value) this took whitened masked GAE 1024 x 2048 from 21.9 to 19.8 us.
template <int kCtrl>
__device__ __forceinline__ double dpp_move_f64(double v) {
    const uint64_t u = __double_as_longlong(v);
    const uint32_t lo = uint32_t(__builtin_amdgcn_update_dpp(0, int(uint32_t(u)), kCtrl, 0xf, 0xf, false));
    const uint32_t hi = uint32_t(__builtin_amdgcn_update_dpp(0, int(uint32_t(u >> 32)), kCtrl, 0xf, 0xf, false));
    return __longlong_as_double((uint64_t(hi) << 32) | lo);
}
__device__ __forceinline__ double read_lane_f64(double v, int lane) {
    const uint64_t u = __double_as_longlong(v);
    const uint32_t lo = uint32_t(__builtin_amdgcn_readlane(int(uint32_t(u)), lane));
    const uint32_t hi = uint32_t(__builtin_amdgcn_readlane(int(uint32_t(u >> 32)), lane));
    return __longlong_as_double((uint64_t(hi) << 32) | lo);
}
__device__ __forceinline__ double wave_sum(double x) {
    x += dpp_move_f64<kDppRowShr + 1>(x);
    x += dpp_move_f64<kDppRowShr + 2>(x);
    x += dpp_move_f64<kDppRowShr + 4>(x);
    x += dpp_move_f64<kDppRowShr + 8>(x);
    return (read_lane_f64(x, 15) + read_lane_f64(x, 31)) + (read_lane_f64(x, 47) + read_lane_f64(x, 63));
}

// Step 1 of one chunk [chunk_lo, chunk_hi) of a workgroup's range [lo, hi) (lane l of wave w
// owns the (63-l)-th group of K steps of the wave's span).
template <typename DT, int K, bool TR, bool HM>
__device__ __forceinline__ void masked_chunk_load(MaskedChunk<DT, K, TR, HM>& c, const MaskedArgs& ma,
                                                  const RowBase& base, int64_t lo, int64_t hi,
                                                  int64_t chunk_lo, int64_t chunk_hi, bool can_full,
                                                  int lane, int wave) {
    const Args& a = ma.a;
    c.p0 = chunk_lo + (int64_t(wave) * kWave + (kWave - 1 - lane)) * K;
    const bool full = can_full && chunk_lo >= lo && chunk_hi <= hi;
    if (full) {
        c.load_full(ma, base, MaskedChunk<DT, K, TR, HM>::kAll);
    } else if (can_full) {
        // lane by lane: vector loads wherever the lane's K steps lie inside the array (the
        // steps outside the range masked off), element-wise otherwise
        constexpr uint32_t kAll = MaskedChunk<DT, K, TR, HM>::kAll;
        const int64_t p = c.p0;
        if (p >= lo && p + K <= hi) {
            c.load_full(ma, base, kAll);
        } else if (p + K > lo && p < hi && p >= 0 && p + K <= a.N * a.T) {
            uint32_t m = kAll;
            RowBase b = base;
            if (p < lo) {
                m &= (kAll << uint32_t(lo - p)) & kAll;
                b = RowBase{base.pos - a.T, base.row - 1, base.t};  // the row before
            }
            if (p + K > hi) m &= kAll >> uint32_t(p + K - hi);
            c.load_full(ma, b, m);
        } else {
            c.load_masked(ma, base, lo, hi);
        }
    } else {
        c.load_masked(ma, base, lo, hi);
    }
}

// Rows kernel for masked GAE: workgroup g owns rows [g*R, g*R + R) and walks them in chunks of
// E = W*64*K steps from the end. `wave_local`: every row lies within one wave's span, so no
// carry crosses waves.
template <typename DT, int K, int W, bool VEC, bool TR, bool HM, bool STATS>
__global__ void __launch_bounds__(W * kWave) masked_gae_kernel(MaskedArgs ma, int64_t rows_per_wg,
                                                               int wave_local) {
    const Args& a = ma.a;
    constexpr int64_t E = int64_t(W) * kWave * K;
    __shared__ float s_m[5][W];
    __shared__ float s_cA, s_cW;
    __shared__ double s_stat[3][W];
    __shared__ f32x4 s_out[K == 8 ? W : 1][K == 8 ? 2 * kWave : 1];
    const int lane = threadIdx.x & (kWave - 1), wave = threadIdx.x / kWave;
    const int64_t row_lo = int64_t(blockIdx.x) * rows_per_wg;
    const int64_t row_hi = min(row_lo + rows_per_wg, a.N);
    const int64_t lo = row_lo * a.T, hi = row_hi * a.T;
    const bool can_full = VEC && a.T >= K;
    const RowBase base{lo, row_lo, 0};
    AW carry{0.f, 0.f};
    double n = 0.0, s1 = 0.0, s2 = 0.0;
    int64_t chunk_hi = (hi + K - 1) / K * K;
    for (;;) {
        const int64_t chunk_lo = chunk_hi - E;
        MaskedChunk<DT, K, TR, HM> c;
        c.oslot = s_out[K == 8 ? wave : 0];
        masked_chunk_load(c, ma, base, lo, hi, chunk_lo, chunk_hi, can_full, lane, wave);
        const Tri incl = c.local(a.p, lane);
        Tri win = identity_tri();
        if (!wave_local) {
            if (lane == kWave - 1) {
                s_m[0][wave] = incl.p; s_m[1][wave] = incl.q; s_m[2][wave] = incl.s;
                s_m[3][wave] = incl.ca; s_m[4][wave] = incl.cw;
            }
            __syncthreads();
            for (int w = W - 1; w > wave; --w)
                win = compose(Tri{s_m[0][w], s_m[1][w], s_m[2][w], s_m[3][w], s_m[4][w]}, win);
        }
        const AW first = c.template finish<STATS>(a, apply(win, carry), can_full, n, s1, s2);
        if (chunk_lo <= lo) break;
        // the next chunk (earlier in time) continues from the state at chunk_lo, held by lane
        // 63 of wave 0
        if (threadIdx.x == kWave - 1) { s_cA = first.A; s_cW = first.W; }
        __syncthreads();
        carry = AW{s_cA, s_cW};
        chunk_hi = chunk_lo;
    }
    if constexpr (STATS) {
        n = wave_sum(n);
        s1 = wave_sum(s1);
        s2 = wave_sum(s2);
        if (lane == 0) { s_stat[0][wave] = n; s_stat[1][wave] = s1; s_stat[2][wave] = s2; }
        __syncthreads();
        if (threadIdx.x == 0) {
            Moments m{0.0, 0.0, 0.0, 0.0};
            for (int w = 0; w < W; ++w) { m.n += s_stat[0][w]; m.s1 += s_stat[1][w]; m.s2 += s_stat[2][w]; }
            ma.partials[blockIdx.x] = m;
        }
    }
}

// Sum of partials [lo, hi) over a workgroup of kNormThreads threads, in one fixed order
// (thread-serial over a stride of kNormThreads, a butterfly within each wave, then the waves in
// order), returned to every thread. Every thread of the workgroup must call it.
constexpr int kNormThreads = 256;

__device__ __forceinline__ Moments sum_partials(const Moments* part, int64_t lo, int64_t hi) {
    __shared__ double s_sum[3][kNormThreads / kWave];
    double n = 0.0, s1 = 0.0, s2 = 0.0;
    constexpr int kBatch = 4;  // partials per thread in flight
    for (int64_t g0 = lo + threadIdx.x; g0 < hi; g0 += int64_t(kBatch) * kNormThreads) {
        Moments m[kBatch];
#pragma unroll
        for (int u = 0; u < kBatch; ++u) {
            const int64_t g = g0 + int64_t(u) * kNormThreads;
            m[u] = g < hi ? part[g] : Moments{0.0, 0.0, 0.0, 0.0};
        }
#pragma unroll
        for (int u = 0; u < kBatch; ++u) { n += m[u].n; s1 += m[u].s1; s2 += m[u].s2; }
    }
    n = wave_sum(n);
    s1 = wave_sum(s1);
    s2 = wave_sum(s2);
    const int wave = threadIdx.x / kWave;
    if ((threadIdx.x & (kWave - 1)) == 0) { s_sum[0][wave] = n; s_sum[1][wave] = s1; s_sum[2][wave] = s2; }
    __syncthreads();
    Moments t{0.0, 0.0, 0.0, 0.0};
#pragma unroll
    for (int w = 0; w < kNormThreads / kWave; ++w) { t.n += s_sum[0][w]; t.s1 += s_sum[1][w]; t.s2 += s_sum[2][w]; }
    return t;
}

// Second-level partials: workgroup j adds partials [j * kDirectPartials, (j + 1) * kDirectPartials).
__global__ void __launch_bounds__(kNormThreads) masked_sum_partials_kernel(const Moments* part,
                                                                           int64_t G, Moments* out) {
    const int64_t lo = int64_t(blockIdx.x) * kDirectPartials;
    const Moments t = sum_partials(part, lo, min(lo + kDirectPartials, G));
    if (threadIdx.x == 0) out[blockIdx.x] = t;
}

// adv <- (adv - mean) * rstd over all `total` elements, mean and rstd from the sum of the G
// partials. Each thread rewrites kNormVec 16-byte vectors (strided by the workgroup size, so
// that a wave's accesses are contiguous), its loads issued before the partials are added up;
// workgroup 0 also does the elements past the last vector and stores {mean, rstd} to `stats`.
// The element-wise form is for advantages not 16-byte aligned.
constexpr int kNormVec = 4;

__device__ __forceinline__ void whitening(const Moments* part, int64_t G, float eps, double* stats,
                                          float& mean, float& rstd) {
    const Moments t = sum_partials(part, 0, G);
    const double m = t.n > 0.0 ? t.s1 / t.n : 0.0;
    const double var = t.n > 1.0 ? fmax(t.s2 - t.s1 * m, 0.0) / (t.n - 1.0) : 0.0;
    const double r = 1.0 / sqrt(var + double(eps));
    if (blockIdx.x == 0 && threadIdx.x == 0) { stats[0] = m; stats[1] = r; }
    mean = float(m);
    rstd = float(r);
}

__global__ void __launch_bounds__(kNormThreads) masked_normalize_kernel(float* adv, int64_t total,
                                                                        const Moments* part,
                                                                        int64_t G, float eps,
                                                                        double* stats, int vec) {
    float mean, rstd;
    const int64_t base = int64_t(blockIdx.x) * kNormThreads * kNormVec + threadIdx.x;
    if (vec) {
        f32x4* p = reinterpret_cast<f32x4*>(adv);
        const int64_t nv = total / 4;
        f32x4 x[kNormVec];
#pragma unroll
        for (int u = 0; u < kNormVec; ++u) {
            const int64_t i = base + int64_t(u) * kNormThreads;
            if (i < nv) x[u] = __builtin_nontemporal_load(p + i);
        }
        whitening(part, G, eps, stats, mean, rstd);
#pragma unroll
        for (int u = 0; u < kNormVec; ++u) {
            const int64_t i = base + int64_t(u) * kNormThreads;
            if (i < nv) __builtin_nontemporal_store((x[u] - mean) * rstd, p + i);
        }
        if (blockIdx.x == 0 && threadIdx.x < total - nv * 4) {
            const int64_t i = nv * 4 + threadIdx.x;
            adv[i] = (adv[i] - mean) * rstd;
        }
    } else {
        // the same 4 * kNormVec * kNormThreads elements per workgroup, one at a time
        const int64_t first = int64_t(blockIdx.x) * kNormThreads * kNormVec * 4 + threadIdx.x;
        float x[4 * kNormVec];
#pragma unroll
        for (int u = 0; u < 4 * kNormVec; ++u) {
            const int64_t i = first + int64_t(u) * kNormThreads;
            if (i < total) x[u] = adv[i];
        }
        whitening(part, G, eps, stats, mean, rstd);
#pragma unroll
        for (int u = 0; u < 4 * kNormVec; ++u) {
            const int64_t i = first + int64_t(u) * kNormThreads;
            if (i < total) adv[i] = (x[u] - mean) * rstd;
        }
    }
}

// ---------------------------------------------------------------- whitening in one pass
// When every workgroup of a whitened call is resident on the GPU at once and holds one chunk,
// the call runs as one kernel: each workgroup computes its advantages, stores the returns,
// keeps the advantages in registers and publishes its fp64 moments; workgroup 0 adds them all
// up (one record per lane, at most one per lane of its W waves) into the mean and
// 1/sqrt(var + eps) and publishes them in kStatsCopies copies; every other workgroup waits for
// its copy; then each whitens its advantages and stores them, once. Two round trips through
// memory follow the last moments. The sums run in one fixed order, so results are
// reproducible bit for bit. Every wait is for a workgroup that is already resident (the host
// launches this form only when the whole grid fits on the GPU at once), and no atomic
// read-modify-write is used (a counter that every workgroup increments serializes them, about
// 17 ns each). A waiting workgroup polls one record with one lane, with pauses that grow, so
// that the waiting workgroups do not flood memory while others still stream their data (every
// workgroup polling every record it needs slowed whole calls several times over).
//
// Workspace of the whitening (zero-filled once before its first use; every call leaves it
// ready for the next):
//   [0, 16)    mean and 1/sqrt(var + eps) of the last call, two doubles (for the caller);
//   [16, 24)   generation: the number of one-pass calls made on the workspace (mod 2^31);
//              workgroup 0 advances it once every moment of its call is in, hence after every
//              workgroup of the call has read it;
//   kMaskedFusedOff: one tagged moments record (six words) per workgroup, kFusedMaxGroups;
//   kMaskedStatsOff: kStatsCopies copies of the tagged statistics record (four words), one per
//              128-byte line;
//   kMaskedTwoPassOff: the partials of the two-pass form (Moments, 32 bytes each).
// A tagged word holds a 32-bit half of a double in its low half and the tag 2*gen + 1 of its
// call in the high half; a reader takes a double only when both of its words carry the
// current tag, so no word of another call (or of the two-pass partials, which live apart)
// passes for a current one. Polls are bounded (the loads may see a write late); on exhaustion
// the statistics are NaN.
constexpr int64_t kFusedMaxGroups = 1024;
constexpr int kStatsCopies = 64;
constexpr size_t kMaskedGenOff = 16;
constexpr size_t kMaskedFusedOff = 64;
constexpr size_t kMaskedStatsOff = (kMaskedFusedOff + 48 * size_t(kFusedMaxGroups) + 127) / 128 * 128;
constexpr size_t kMaskedTwoPassOff = kMaskedStatsOff + 128 * size_t(kStatsCopies);

__device__ __forceinline__ void put_tagged(uint64_t* w, double v, uint32_t tag) {
    const uint64_t u = uint64_t(__double_as_longlong(v));
    st_relaxed(w, uint64_t(tag) << 32 | (u & 0xffffffffu));
    st_relaxed(w + 1, uint64_t(tag) << 32 | (u >> 32));
}

// Doubles v[0 .. M) from the tagged words w[0 .. 2M) once every word carries `tag`: all words
// are loaded at once and reloaded until they do, after a pause that doubles from `pause`
// to about 500 cycles (NaN after kMaxPolls rounds).
template <int M>
__device__ __forceinline__ void get_tagged(const uint64_t* w, uint32_t tag, double (&v)[M], int pause) {
    uint64_t x[2 * M];
#pragma unroll
    for (int i = 0; i < 2 * M; ++i) x[i] = ld_relaxed(w + i);
    for (uint32_t polls = 0;; ++polls) {
        bool ok = true;
#pragma unroll
        for (int i = 0; i < 2 * M; ++i) ok = ok && uint32_t(x[i] >> 32) == tag;
        if (ok) break;
        if (polls >= kMaxPolls) {
#pragma unroll
            for (int i = 0; i < M; ++i) v[i] = __builtin_nan("");
            return;
        }
        for (int i = 0; i < pause; ++i) __builtin_amdgcn_s_sleep(2);
        pause = min(2 * pause, 4);
        // every word again, all loads in flight together: a word that already carried the tag
        // carries it still (each word of a record is written once per call)
#pragma unroll
        for (int i = 0; i < 2 * M; ++i) x[i] = ld_relaxed(w + i);
    }
#pragma unroll
    for (int i = 0; i < M; ++i)
        v[i] = __longlong_as_double(int64_t((x[2 * i + 1] << 32) | (x[2 * i] & 0xffffffffu)));
}

// One-pass whitened masked GAE: workgroup g owns rows [g*R, g*R + R), which fit in one chunk;
// every workgroup of the grid (G <= W * 64 <= kFusedMaxGroups of them) is resident at once.
// `ws`: the whitening workspace.
template <typename DT, int K, int W, bool VEC, bool TR, bool HM>
__global__ void __launch_bounds__(W * kWave) masked_gae_fused_kernel(MaskedArgs ma, int64_t rows_per_wg,
                                                                     int wave_local, float eps,
                                                                     char* ws) {
    static_assert(int64_t(W) * kWave <= kFusedMaxGroups, "one moments record per lane of workgroup 0");
    const Args& a = ma.a;
    constexpr int64_t E = int64_t(W) * kWave * K;
    __shared__ float s_m[5][W];
    __shared__ double s_stat[3][W];
    __shared__ uint32_t s_tag;
    __shared__ float s_mean, s_rstd;
    __shared__ f32x4 s_out[K == 8 ? W : 1][K == 8 ? 2 * kWave : 1];
    const int lane = threadIdx.x & (kWave - 1), wave = threadIdx.x / kWave;
    const int64_t G = gridDim.x, g = blockIdx.x;
    const int64_t row_lo = g * rows_per_wg;
    const int64_t row_hi = min(row_lo + rows_per_wg, a.N);
    const int64_t lo = row_lo * a.T, hi = row_hi * a.T;
    const bool can_full = VEC && a.T >= K;
    const RowBase base{lo, row_lo, 0};
    const int64_t chunk_hi = (hi + K - 1) / K * K;
    const int64_t chunk_lo = chunk_hi - E;  // <= lo: the rows fit in one chunk
    uint64_t* gen_word = reinterpret_cast<uint64_t*>(ws + kMaskedGenOff);
    uint64_t* rec = reinterpret_cast<uint64_t*>(ws + kMaskedFusedOff);
    uint64_t* stats_rec = reinterpret_cast<uint64_t*>(ws + kMaskedStatsOff);
    // the generation cannot move before this workgroup's moments are in
    if (threadIdx.x == 0) s_tag = 2u * (uint32_t(ld_relaxed(gen_word)) & 0x7fffffffu) + 1u;

    MaskedChunk<DT, K, TR, HM> c;
    c.oslot = s_out[K == 8 ? wave : 0];
    masked_chunk_load(c, ma, base, lo, hi, chunk_lo, chunk_hi, can_full, lane, wave);
    const Tri incl = c.local(a.p, lane);
    Tri win = identity_tri();
    if (!wave_local) {
        if (lane == kWave - 1) {
            s_m[0][wave] = incl.p; s_m[1][wave] = incl.q; s_m[2][wave] = incl.s;
            s_m[3][wave] = incl.ca; s_m[4][wave] = incl.cw;
        }
        __syncthreads();
        for (int w = W - 1; w > wave; --w)
            win = compose(Tri{s_m[0][w], s_m[1][w], s_m[2][w], s_m[3][w], s_m[4][w]}, win);
    }
    double n = 0.0, s1 = 0.0, s2 = 0.0;
    c.template finish<true, false>(a, apply(win, AW{0.f, 0.f}), can_full, n, s1, s2);

    // this workgroup's moments
    n = wave_sum(n);
    s1 = wave_sum(s1);
    s2 = wave_sum(s2);
    if (lane == 0) { s_stat[0][wave] = n; s_stat[1][wave] = s1; s_stat[2][wave] = s2; }
    __syncthreads();
    const uint32_t tag = s_tag;
    if (g != 0) {
        if (threadIdx.x == 0) {
            Moments m{0.0, 0.0, 0.0, 0.0};
            for (int w = 0; w < W; ++w) { m.n += s_stat[0][w]; m.s1 += s_stat[1][w]; m.s2 += s_stat[2][w]; }
            uint64_t* mine = rec + 6 * g;
            put_tagged(mine, m.n, tag);
            put_tagged(mine + 2, m.s1, tag);
            put_tagged(mine + 4, m.s2, tag);
            double v[2];
            get_tagged<2>(stats_rec + 16 * (g % kStatsCopies), tag, v, 2);
            s_mean = float(v[0]);
            s_rstd = float(v[1]);
        }
    } else {
        // workgroup 0: every workgroup's moments (its own from LDS), one per lane
        double v[3] = {0.0, 0.0, 0.0};
        if (threadIdx.x == 0) {
            for (int w = 0; w < W; ++w) { v[0] += s_stat[0][w]; v[1] += s_stat[1][w]; v[2] += s_stat[2][w]; }
        } else if (threadIdx.x < G) {
            get_tagged<3>(rec + 6 * int64_t(threadIdx.x), tag, v, 1);
        }
        __syncthreads();  // every lane of workgroup 0 has read s_stat
        v[0] = wave_sum(v[0]);
        v[1] = wave_sum(v[1]);
        v[2] = wave_sum(v[2]);
        if (lane == 0) { s_stat[0][wave] = v[0]; s_stat[1][wave] = v[1]; s_stat[2][wave] = v[2]; }
        __syncthreads();
        if (wave == 0) {
            Moments t{0.0, 0.0, 0.0, 0.0};
            for (int w = 0; w < W; ++w) { t.n += s_stat[0][w]; t.s1 += s_stat[1][w]; t.s2 += s_stat[2][w]; }
            const double m = t.n > 0.0 ? t.s1 / t.n : 0.0;
            const double var = t.n > 1.0 ? fmax(t.s2 - t.s1 * m, 0.0) / (t.n - 1.0) : 0.0;
            const double r = 1.0 / sqrt(var + double(eps));
            uint64_t* copy = stats_rec + 16 * lane;  // one 128-byte line per copy
            put_tagged(copy, m, tag);
            put_tagged(copy + 2, r, tag);
            if (lane == 0) {
                // every moment of the call is in, so every workgroup has read the generation
                double* stats = reinterpret_cast<double*>(ws);
                stats[0] = m;
                stats[1] = r;
                st_relaxed(gen_word, uint64_t(((tag - 1u) / 2u + 1u) & 0x7fffffffu));
                s_mean = float(m);
                s_rstd = float(r);
            }
        }
    }
    __syncthreads();
    const float mean = s_mean, rstd = s_rstd;
    float y[K];
#pragma unroll
    for (int k = 0; k < K; ++k) y[k] = (c.adv[k] - mean) * rstd;
    c.store(a.out0, can_full && c.valid == MaskedChunk<DT, K, TR, HM>::kAll, y);
}

}  // namespace rlcs
