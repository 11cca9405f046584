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
// workgroup to (count, mean, M2) in fp64; one workgroup merges those partials in a fixed order
// (Chan et al.'s pairwise update) into the mean and 1/sqrt(var + eps), var the unbiased
// variance; a last kernel rewrites the advantages. Every order is fixed, so results are
// reproducible bit for bit.
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

template <int S>
__device__ __forceinline__ Tri tri_row_shr(const Tri& v) {
    return Tri{dpp_move<kDppRowShr + S>(1.f, v.p), dpp_move<kDppRowShr + S>(0.f, v.q),
               dpp_move<kDppRowShr + S>(1.f, v.s), dpp_move<kDppRowShr + S>(0.f, v.ca),
               dpp_move<kDppRowShr + S>(0.f, v.cw)};
}

__device__ __forceinline__ float readlane_f(float v, int lane) {
    return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), lane));
}

__device__ __forceinline__ Tri read_lane(const Tri& v, int lane) {
    return Tri{readlane_f(v.p, lane), readlane_f(v.q, lane), readlane_f(v.s, lane),
               readlane_f(v.ca, lane), readlane_f(v.cw, lane)};
}

// Inclusive prefix scan of per-lane maps over the 64 lanes, as wave_scan_inclusive for pairs.
__device__ __forceinline__ Tri wave_scan_inclusive(Tri v, int lane) {
    v = compose(v, tri_row_shr<1>(v));
    v = compose(v, tri_row_shr<2>(v));
    v = compose(v, tri_row_shr<4>(v));
    v = compose(v, tri_row_shr<8>(v));
    const Tri t0 = read_lane(v, 15), t1 = read_lane(v, 31), t2 = read_lane(v, 47);
    const Tri p2 = compose(t1, t0);
    const Tri p3 = compose(t2, p2);
    const int row = lane >> 4;
    if (row > 0) v = compose(v, (row == 1) ? t0 : ((row == 2) ? p2 : p3));
    return v;
}

// Value of lane l-1 (lane 0 receives `fill`).
__device__ __forceinline__ AW shift_up1(AW v, AW fill) {
    return AW{shift_up1(v.A, fill.A), shift_up1(v.W, fill.W)};
}

struct MaskedArgs {
    Args a;              // in[0] r, in[1] v, in[2] bv; term, trunc; row_value = boot;
                         // out0 adv, out1 ret (optional)
    const uint8_t* mask; // [N, T], nonzero = the step takes part; null = every step does
    double* partials;    // per-workgroup (count, mean, M2) of the advantages that take part
};

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

    // Steps of a chunk whose K steps are all in range, 16-byte aligned data and T >= K: vector
    // loads, every one issued before the first use; at most one row edge.
    __device__ __forceinline__ void load_full(const MaskedArgs& ma, const RowBase& base) {
        const Args& a = ma.a;
        valid = kAll;
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
    // first step. Accumulates the advantages that take part into (n, sum, sumsq).
    template <bool STATS>
    __device__ __forceinline__ AW finish(const Args& a, AW Xw, bool full, double& n, double& s1,
                                         double& s2) {
        AW x = shift_up1(apply(incl, Xw), Xw);
        float adv[K], ret[K];
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
        store_k<K>(a.out0, p0, valid, full, adv);
        if (a.out1) store_k<K>(a.out1, p0, valid, full, ret);
        return x;
    }
};

__device__ __forceinline__ double wave_sum(double x) {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) x += __shfl_xor(x, o, kWave);
    return x;
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
        c.p0 = chunk_lo + (int64_t(wave) * kWave + (kWave - 1 - lane)) * K;
        const bool full = can_full && chunk_lo >= lo && chunk_hi <= hi;
        if (full) c.load_full(ma, base);
        else c.load_masked(ma, base, lo, hi);
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
        const AW first = c.template finish<STATS>(a, apply(win, carry), full, n, s1, s2);
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
            double tn = 0.0, t1 = 0.0, t2 = 0.0;
            for (int w = 0; w < W; ++w) { tn += s_stat[0][w]; t1 += s_stat[1][w]; t2 += s_stat[2][w]; }
            const double mean = tn > 0.0 ? t1 / tn : 0.0;
            const double m2 = tn > 0.0 ? fmax(t2 - t1 * mean, 0.0) : 0.0;
            double* out = ma.partials + 4 * int64_t(blockIdx.x);
            out[0] = tn;
            out[1] = mean;
            out[2] = m2;
        }
    }
}

// One workgroup: merges the G partials (count, mean, M2) in a fixed order and writes the mean
// and 1/sqrt(var + eps) (var unbiased; 0 with fewer than two advantages) to stats[0..1].
constexpr int kReduceThreads = 1024;

__global__ void __launch_bounds__(kReduceThreads) masked_stats_kernel(const double* partials,
                                                                      int64_t G, float eps,
                                                                      double* stats) {
    __shared__ double s_n[kReduceThreads], s_mean[kReduceThreads], s_m2[kReduceThreads];
    const int tid = threadIdx.x;
    double n = 0.0, mean = 0.0, m2 = 0.0;
    for (int64_t g = tid; g < G; g += kReduceThreads) {
        const double nb = partials[4 * g], mb = partials[4 * g + 1], m2b = partials[4 * g + 2];
        if (nb == 0.0) continue;
        const double nn = n + nb, d = mb - mean;
        mean += d * (nb / nn);
        m2 += m2b + d * d * (n * nb / nn);
        n = nn;
    }
    s_n[tid] = n; s_mean[tid] = mean; s_m2[tid] = m2;
    __syncthreads();
    for (int half = kReduceThreads / 2; half > 0; half >>= 1) {
        if (tid < half) {
            const double na = s_n[tid], nb = s_n[tid + half];
            if (nb > 0.0) {
                const double nn = na + nb, d = s_mean[tid + half] - s_mean[tid];
                s_mean[tid] += d * (nb / nn);
                s_m2[tid] += s_m2[tid + half] + d * d * (na * nb / nn);
                s_n[tid] = nn;
            }
        }
        __syncthreads();
    }
    if (tid == 0) {
        const double var = s_n[0] > 1.0 ? s_m2[0] / (s_n[0] - 1.0) : 0.0;
        stats[0] = s_n[0] > 0.0 ? s_mean[0] : 0.0;
        stats[1] = 1.0 / sqrt(var + double(eps));
    }
}

// adv <- (adv - mean) * rstd over all `total` elements (grid-stride, 16-byte vectors when
// aligned).
__global__ void __launch_bounds__(256) masked_normalize_kernel(float* adv, int64_t total,
                                                               const double* stats, int vec) {
    const float mean = float(stats[0]), rstd = float(stats[1]);
    const int64_t stride = int64_t(gridDim.x) * blockDim.x;
    const int64_t tid = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
    if (vec) {
        f32x4* p = reinterpret_cast<f32x4*>(adv);
        const int64_t nv = total / 4;
        for (int64_t i = tid; i < nv; i += stride) {
            f32x4 x = __builtin_nontemporal_load(p + i);
            x = (x - mean) * rstd;
            __builtin_nontemporal_store(x, p + i);
        }
        for (int64_t i = nv * 4 + tid; i < total; i += stride) adv[i] = (adv[i] - mean) * rstd;
    } else {
        for (int64_t i = tid; i < total; i += stride) adv[i] = (adv[i] - mean) * rstd;
    }
}

}  // namespace rlcs
