// Per-estimator coefficient builders (Table 1 with the boundary rules of Section 3.2) and
// epilogues. Each policy describes:
//   kBackward   direction of its recurrence (Section 1, Eq. 1);
//   kSlots      number of [N, T] data inputs it reads (Args::in[0 .. kSlots-1]);
//   slot_used   whether slot s is read (the truncation continuation only with truncation);
//   kTruncSlot  the slot read only at truncated steps (-1: none); a lane loads it only when
//               one of its steps is truncated;
//   kFlags      whether it reads term / trunc;
//   kRowValue   whether it reads the per-row value (bootstrap or carry) at the row edge;
//   kNbr        number of values it needs from the neighbouring step on the carry-source side
//               (exported by that step's lane, or at a wave edge loaded raw from memory by
//               nbr_load_raw and converted by nbr_fix once every load has been issued);
//   build       alpha_k, beta_k of the lane's K steps;
//   finish      the outputs of the K steps given the scanned values A_k and X, the scanned
//               value just past the lane on the carry-source side.
//
// Row edges are folded into the coefficients so that one segmented scan runs over the flat
// [N*T] array: at the last step of a row (backward) or the first (forward) beta is 0, and a
// nonzero carry A_T (or z_{-1}) enters alpha as beta * carry, which equals adding
// decay_product * carry after the scan (Section 4.1, step 4).
#pragma once

#include "rlcs_device.h"

namespace rlcs {

struct Params {
    float gamma, lambda, rho_bar, c_bar;
};

struct Args {
    const void* in[5];     // data inputs, meaning fixed by the policy
    const int32_t* actions;  // full-form Retrace: taken actions [N, T]
    int64_t A;             // full-form Retrace: number of actions
    int64_t A_slice;       // full-form Retrace, long action axes: actions staged at a time
    int stage_vec;         // full-form Retrace: Q and pi are 16-byte aligned
    const uint8_t* term;   // [N, T] or null
    const uint8_t* trunc;  // [N, T] or null
    const void* row_value; // [N] bootstrap / carry, or null (= 0)
    float* out0;
    float* out1;           // may be null
    Params p;
    int64_t N, T;
    float inv_T;           // 1 / T in fp32 (row bookkeeping)
    // Positions of the rows kernel: row n's step t at n * period + t (period = T for dense
    // rows; a row stride above T for strided rows, whose steps t >= T are not part of the
    // call and are neither read nor written).
    int64_t period;
    float inv_period;
    void* ws;              // cross-workgroup carry records (split-row variant only)
};

// Defaults shared by the policies: no inputs staged through LDS.
struct OpBase {
    static constexpr int kStaged = 0;
    static constexpr bool kSliced = false;  // staged policies: action axis taken in slices
    static constexpr int staged_index(int) { return -1; }
};

// Bit helpers over K-bit masks.
__device__ __forceinline__ bool bit(uint32_t m, int k) { return (m >> k) & 1u; }

// Successor value of step k as Section 3.2 defines it: 0 after a termination, the supplied
// continuation after a truncation, the row bootstrap at the window edge, else the next
// step's value.
__device__ __forceinline__ float successor(bool term, bool trunc, bool edge, float bv, float B,
                                           float next) {
    return term ? 0.f : (trunc ? bv : (edge ? B : next));
}

// ---------------------------------------------------------------- GAE (Section 3.3.1)
// in: r, v, bv
struct GaeOp : OpBase {
    static constexpr bool kBackward = true;
    static constexpr int kSlots = 3;
    static constexpr int kTruncSlot = 2;  // read only at truncated steps
    static constexpr bool kFlags = true, kRowValue = true;
    static constexpr int kNbr = 1;  // V of the next step
    static constexpr bool slot_used(int s, bool trunc) { return s < 2 || trunc; }

    template <int K>
    __device__ static void nbr_export(const Params&, const float (&d)[kSlots][K], uint32_t, float (&nb)[kNbr]) {
        nb[0] = d[1][0];
    }
    static constexpr int kNbrRaw = kNbr;
    template <typename DT>
    __device__ static void nbr_load_raw(const Args& a, int64_t p, float (&raw)[kNbrRaw]) {
        raw[0] = load_one<DT>(a.in[1], p);
    }
    __device__ static void nbr_fix(const Args&, const float (&raw)[kNbrRaw], float (&nb)[kNbr]) {
        nb[0] = raw[0];
    }
    template <int K, bool TR>
    __device__ static void build(const Params& P, const float (&d)[kSlots][K], uint32_t term,
                                 uint32_t trunc, uint32_t edge, const float (&B)[K],
                                 const float (&nb)[kNbr], float (&al)[K], float (&be)[K]) {
        const float gl = P.gamma * P.lambda;
#pragma unroll
        for (int k = 0; k < K; ++k) {
            const bool te = bit(term, k), tr = TR && bit(trunc, k), ed = bit(edge, k);
            const float next = (k + 1 < K) ? d[1][k + 1] : nb[0];
            const float s = successor(te, tr, ed, TR ? d[2][k] : 0.f, B[k], next);
            al[k] = fmaf(P.gamma, s, d[0][k]) - d[1][k];
            be[k] = (te || tr || ed) ? 0.f : gl;
        }
    }
    template <int K, bool TR>
    __device__ static void finish(const Params&, const float (&d)[kSlots][K], uint32_t, uint32_t,
                                  uint32_t, const float (&)[K], const float (&)[kNbr],
                                  const float (&A)[K], float, float (&o0)[K], float (&o1)[K]) {
#pragma unroll
        for (int k = 0; k < K; ++k) { o0[k] = A[k]; o1[k] = A[k] + d[1][k]; }
    }
};

// ---------------------------------------------------------------- V-Trace (Section 3.3.2)
// in: r, v, log_rho, bv
struct VtraceOp : OpBase {
    static constexpr bool kBackward = true;
    static constexpr int kSlots = 4;
    static constexpr int kTruncSlot = 3;  // read only at truncated steps
    static constexpr bool kFlags = true, kRowValue = true;
    static constexpr int kNbr = 1;  // V of the next step
    static constexpr bool slot_used(int s, bool trunc) { return s < 3 || trunc; }

    template <int K>
    __device__ static void nbr_export(const Params&, const float (&d)[kSlots][K], uint32_t, float (&nb)[kNbr]) {
        nb[0] = d[1][0];
    }
    static constexpr int kNbrRaw = kNbr;
    template <typename DT>
    __device__ static void nbr_load_raw(const Args& a, int64_t p, float (&raw)[kNbrRaw]) {
        raw[0] = load_one<DT>(a.in[1], p);
    }
    __device__ static void nbr_fix(const Args&, const float (&raw)[kNbrRaw], float (&nb)[kNbr]) {
        nb[0] = raw[0];
    }
    template <int K, bool TR>
    __device__ static void build(const Params& P, const float (&d)[kSlots][K], uint32_t term,
                                 uint32_t trunc, uint32_t edge, const float (&B)[K],
                                 const float (&nb)[kNbr], float (&al)[K], float (&be)[K]) {
#pragma unroll
        for (int k = 0; k < K; ++k) {
            const bool te = bit(term, k), tr = TR && bit(trunc, k), ed = bit(edge, k);
            const float ratio = __expf(d[2][k]);
            const float rho = fminf(P.rho_bar, ratio);
            const float c = fminf(P.c_bar, ratio);
            const float next = (k + 1 < K) ? d[1][k + 1] : nb[0];
            const float s = successor(te, tr, ed, TR ? d[3][k] : 0.f, B[k], next);
            al[k] = rho * (fmaf(P.gamma, s, d[0][k]) - d[1][k]);
            be[k] = (te || tr || ed) ? 0.f : P.gamma * c;
        }
    }
    template <int K, bool TR>
    __device__ static void finish(const Params& P, const float (&d)[kSlots][K], uint32_t term,
                                  uint32_t trunc, uint32_t edge, const float (&B)[K],
                                  const float (&nb)[kNbr], const float (&A)[K], float X,
                                  float (&o0)[K], float (&o1)[K]) {
#pragma unroll
        for (int k = 0; k < K; ++k) {
            const bool te = bit(term, k), tr = TR && bit(trunc, k), ed = bit(edge, k);
            const float rho = fminf(P.rho_bar, __expf(d[2][k]));
            // vs of the next step: V_{t+1} + Delta_{t+1}
            const float vs_next = (k + 1 < K) ? d[1][k + 1] + A[k + 1] : nb[0] + X;
            const float s = successor(te, tr, ed, TR ? d[3][k] : 0.f, B[k], vs_next);
            o0[k] = d[1][k] + A[k];
            o1[k] = rho * (fmaf(P.gamma, s, d[0][k]) - d[1][k]);
        }
    }
};

// ---------------------------------------------------------------- Retrace (Section 3.3.3)
// in: r, q, eq, log_rho, bv
struct RetraceOp : OpBase {
    static constexpr bool kBackward = true;
    static constexpr int kSlots = 5;
    static constexpr int kTruncSlot = 4;  // read only at truncated steps
    static constexpr bool kFlags = true, kRowValue = true;
    static constexpr int kNbr = 2;  // E_pi Q and c of the next step
    static constexpr bool slot_used(int s, bool trunc) { return s < 4 || trunc; }

    __device__ static float trace(const Params& P, float log_rho) {
        return P.lambda * fminf(P.c_bar, __expf(log_rho));
    }
    template <int K>
    __device__ static void nbr_export(const Params& P, const float (&d)[kSlots][K], uint32_t, float (&nb)[kNbr]) {
        nb[0] = d[2][0];
        nb[1] = trace(P, d[3][0]);
    }
    static constexpr int kNbrRaw = kNbr;
    template <typename DT>
    __device__ static void nbr_load_raw(const Args& a, int64_t p, float (&raw)[kNbrRaw]) {
        raw[0] = load_one<DT>(a.in[2], p);
        raw[1] = load_one<DT>(a.in[3], p);
    }
    __device__ static void nbr_fix(const Args& a, const float (&raw)[kNbrRaw], float (&nb)[kNbr]) {
        nb[0] = raw[0];
        nb[1] = trace(a.p, raw[1]);
    }
    template <int K, bool TR>
    __device__ static void build(const Params& P, const float (&d)[kSlots][K], uint32_t term,
                                 uint32_t trunc, uint32_t edge, const float (&B)[K],
                                 const float (&nb)[kNbr], float (&al)[K], float (&be)[K]) {
#pragma unroll
        for (int k = 0; k < K; ++k) {
            const bool te = bit(term, k), tr = TR && bit(trunc, k), ed = bit(edge, k);
            const float eq_next = (k + 1 < K) ? d[2][k + 1] : nb[0];
            const float c_next = (k + 1 < K) ? trace(P, d[3][k + 1]) : nb[1];
            const float s = successor(te, tr, ed, TR ? d[4][k] : 0.f, B[k], eq_next);
            al[k] = fmaf(P.gamma, s, d[0][k]) - d[1][k];
            // c_T = 0: the last step of a row never carries (edge)
            be[k] = (te || tr || ed) ? 0.f : P.gamma * c_next;
        }
    }
    template <int K, bool TR>
    __device__ static void finish(const Params&, const float (&d)[kSlots][K], uint32_t, uint32_t,
                                  uint32_t, const float (&)[K], const float (&)[kNbr],
                                  const float (&A)[K], float, float (&o0)[K], float (&o1)[K]) {
#pragma unroll
        for (int k = 0; k < K; ++k) { o0[k] = A[k]; o1[k] = d[1][k] + A[k]; }
    }
};

// ---------------------------------------------------------------- full-form Retrace (Section 7.3)
// Global inputs: in[0] r, in[4] bv (truncated steps only); the [N, T, A] Q-values in[1] and
// target probabilities in[2], the taken actions and the behaviour probabilities in[3] are
// reduced per step while the chunk is staged, into three LDS slots:
//   slot 1: Q(s_t, a_t),  slot 2: E_pi Q(s_t) = sum_a pi(a|s_t) Q(s_t, a),
//   slot 3: rho_t = pi(a_t|s_t) / mu(a_t|s_t).
// An action outside [0, A) selects nothing (Q and pi taken as 0). The recurrence is
// RetraceOp's with c_t = lambda * min(c_bar, rho_t).
struct RetraceFullOp : OpBase {
    static constexpr bool kBackward = true;
    static constexpr int kSlots = 5;
    static constexpr int kTruncSlot = 4;  // read only at truncated steps
    static constexpr bool kFlags = true, kRowValue = true;
    static constexpr int kNbr = 2;  // E_pi Q and c of the next step, read from the stage
    static constexpr int kNbrRaw = 1;
    static constexpr int kStaged = 3;
    static constexpr int staged_index(int s) { return (s >= 1 && s <= 3) ? s - 1 : -1; }
    static constexpr bool slot_used(int s, bool trunc) { return s == 0 || (s == 4 && trunc); }

    __device__ static float trace(const Params& P, float rho) { return P.lambda * fminf(P.c_bar, rho); }

    // Staged terms of one step from its rows Q(s_t, .) and pi(.|s_t) (in LDS), its action and
    // its behaviour probability: v = {Q(s_t, a_t), E_pi Q(s_t), rho_t}. The expectation sums
    // the actions in order. `rows16`: both rows start on 16-byte boundaries and hold whole
    // 16-byte blocks, read one block at a time. An action outside [0, A) selects nothing.
    template <typename DT>
    __device__ __forceinline__ static void reduce_step(const DT* q_row, const DT* pi_row, int64_t A, bool rows16,
                                       int32_t act, float mu, float (&v)[kStaged]) {
        constexpr int kPer = 16 / int(sizeof(DT));
        float e = 0.f, qa = 0.f, pa = 0.f;
        if (rows16) {
            for (int64_t b = 0; b < A / kPer; ++b) {
                const u32x4 bq = *reinterpret_cast<const u32x4*>(q_row + b * kPer);
                const u32x4 bp = *reinterpret_cast<const u32x4*>(pi_row + b * kPer);
#pragma unroll
                for (int u = 0; u < kPer; ++u) {
                    const float qk = word_elem<DT>(bq[u * 4 / kPer], u);
                    const float pk = word_elem<DT>(bp[u * 4 / kPer], u);
                    e = fmaf(pk, qk, e);
                    if (b * kPer + u == act) { qa = qk; pa = pk; }
                }
            }
        } else {
            for (int64_t k = 0; k < A; ++k) {
                const float qk = widen(q_row[k]), pk = widen(pi_row[k]);
                e = fmaf(pk, qk, e);
                if (k == act) { qa = qk; pa = pk; }
            }
        }
        v[0] = qa;
        v[1] = e;
        v[2] = pa / mu;
    }
    // One slice of a step's rows, actions [a0, a0 + aw) (row pointers at action a0): adds
    // pi * Q over the slice to `e`, in action order, and takes Q and pi of the taken action if
    // it lies in the slice. Rows of whole 16-byte blocks are read one block at a time.
    template <typename DT>
    __device__ __forceinline__ static void accumulate_slice(const DT* q_row, const DT* pi_row, int64_t a0,
                                                            int64_t aw, int32_t act, float& e, float& qa,
                                                            float& pa) {
        constexpr int kPer = 16 / int(sizeof(DT));
        if (aw % kPer == 0) {
            for (int64_t b = 0; b < aw / kPer; ++b) {
                const u32x4 bq = *reinterpret_cast<const u32x4*>(q_row + b * kPer);
                const u32x4 bp = *reinterpret_cast<const u32x4*>(pi_row + b * kPer);
#pragma unroll
                for (int u = 0; u < kPer; ++u) {
                    const float qk = word_elem<DT>(bq[u * 4 / kPer], u);
                    const float pk = word_elem<DT>(bp[u * 4 / kPer], u);
                    e = fmaf(pk, qk, e);
                    if (a0 + b * kPer + u == act) { qa = qk; pa = pk; }
                }
            }
        } else {
            for (int64_t k = 0; k < aw; ++k) {
                const float qk = widen(q_row[k]), pk = widen(pi_row[k]);
                e = fmaf(pk, qk, e);
                if (a0 + k == act) { qa = qk; pa = pk; }
            }
        }
    }
    __device__ static void nbr_from_stage(const Params& P, const float* stage, int stride, int i,
                                          float (&nb)[kNbr]) {
        nb[0] = stage[1 * stride + i];
        nb[1] = trace(P, stage[2 * stride + i]);
    }
    template <int K>
    __device__ static void nbr_export(const Params&, const float (&)[kSlots][K], uint32_t, float (&)[kNbr]) {}
    template <typename DT>
    __device__ static void nbr_load_raw(const Args&, int64_t, float (&)[kNbrRaw]) {}
    __device__ static void nbr_fix(const Args&, const float (&)[kNbrRaw], float (&)[kNbr]) {}

    template <int K, bool TR>
    __device__ static void build(const Params& P, const float (&d)[kSlots][K], uint32_t term,
                                 uint32_t trunc, uint32_t edge, const float (&B)[K],
                                 const float (&nb)[kNbr], float (&al)[K], float (&be)[K]) {
#pragma unroll
        for (int k = 0; k < K; ++k) {
            const bool te = bit(term, k), tr = TR && bit(trunc, k), ed = bit(edge, k);
            const float eq_next = (k + 1 < K) ? d[2][k + 1] : nb[0];
            const float c_next = (k + 1 < K) ? trace(P, d[3][k + 1]) : nb[1];
            const float s = successor(te, tr, ed, TR ? d[4][k] : 0.f, B[k], eq_next);
            al[k] = fmaf(P.gamma, s, d[0][k]) - d[1][k];
            be[k] = (te || tr || ed) ? 0.f : P.gamma * c_next;
        }
    }
    template <int K, bool TR>
    __device__ static void finish(const Params&, const float (&d)[kSlots][K], uint32_t, uint32_t,
                                  uint32_t, const float (&)[K], const float (&)[kNbr],
                                  const float (&A)[K], float, float (&o0)[K], float (&o1)[K]) {
#pragma unroll
        for (int k = 0; k < K; ++k) { o0[k] = A[k]; o1[k] = d[1][k] + A[k]; }
    }
};

// Full-form Retrace with the action axis staged in slices (axes too long for a chunk's whole
// [steps, A] slices in LDS).
struct RetraceFullSlicedOp : RetraceFullOp {
    static constexpr bool kSliced = true;
};

// ---------------------------------------------------------------- TD(lambda) (Section 3.3.4)
// in: r, v, bv
struct TdLambdaOp : OpBase {
    static constexpr bool kBackward = true;
    static constexpr int kSlots = 3;
    static constexpr int kTruncSlot = 2;  // read only at truncated steps
    static constexpr bool kFlags = true, kRowValue = true;
    static constexpr int kNbr = 1;
    static constexpr bool slot_used(int s, bool trunc) { return s < 2 || trunc; }

    template <int K>
    __device__ static void nbr_export(const Params&, const float (&d)[kSlots][K], uint32_t, float (&nb)[kNbr]) {
        nb[0] = d[1][0];
    }
    static constexpr int kNbrRaw = kNbr;
    template <typename DT>
    __device__ static void nbr_load_raw(const Args& a, int64_t p, float (&raw)[kNbrRaw]) {
        raw[0] = load_one<DT>(a.in[1], p);
    }
    __device__ static void nbr_fix(const Args&, const float (&raw)[kNbrRaw], float (&nb)[kNbr]) {
        nb[0] = raw[0];
    }
    template <int K, bool TR>
    __device__ static void build(const Params& P, const float (&d)[kSlots][K], uint32_t term,
                                 uint32_t trunc, uint32_t edge, const float (&B)[K],
                                 const float (&nb)[kNbr], float (&al)[K], float (&be)[K]) {
        const float gl = P.gamma * P.lambda;
        const float g1l = P.gamma * (1.f - P.lambda);
#pragma unroll
        for (int k = 0; k < K; ++k) {
            const bool te = bit(term, k), tr = TR && bit(trunc, k), ed = bit(edge, k);
            const bool done = te || tr;
            const float next = (k + 1 < K) ? d[1][k + 1] : nb[0];
            float a;
            if (te)       a = d[0][k];                          // no successor value
            else if (tr)  a = fmaf(P.gamma, d[2][k], d[0][k]);  // full-gamma continuation
            else if (ed)  a = fmaf(P.gamma, B[k], d[0][k]);     // gamma(1-l) B + carry gamma l B
            else          a = fmaf(g1l, next, d[0][k]);
            al[k] = a;
            be[k] = (done || ed) ? 0.f : gl;
        }
    }
    template <int K, bool TR>
    __device__ static void finish(const Params&, const float (&)[kSlots][K], uint32_t, uint32_t,
                                  uint32_t, const float (&)[K], const float (&)[kNbr],
                                  const float (&A)[K], float, float (&o0)[K], float (&)[K]) {
#pragma unroll
        for (int k = 0; k < K; ++k) o0[k] = A[k];
    }
};

// ---------------------------------------------------------------- discounted returns (Section 3.3.4)
// in: r, bv
struct DiscountedOp : OpBase {
    static constexpr bool kBackward = true;
    static constexpr int kSlots = 2;
    static constexpr int kTruncSlot = 1;  // read only at truncated steps
    static constexpr bool kFlags = true, kRowValue = true;
    static constexpr int kNbr = 0;
    static constexpr bool slot_used(int s, bool trunc) { return s < 1 || trunc; }

    template <int K>
    __device__ static void nbr_export(const Params&, const float (&)[kSlots][K], uint32_t, float (&)[1]) {}
    static constexpr int kNbrRaw = 1;
    template <typename DT>
    __device__ static void nbr_load_raw(const Args&, int64_t, float (&)[1]) {}
    __device__ static void nbr_fix(const Args&, const float (&)[1], float (&)[1]) {}
    template <int K, bool TR>
    __device__ static void build(const Params& P, const float (&d)[kSlots][K], uint32_t term,
                                 uint32_t trunc, uint32_t edge, const float (&B)[K],
                                 const float (&)[1], float (&al)[K], float (&be)[K]) {
#pragma unroll
        for (int k = 0; k < K; ++k) {
            const bool te = bit(term, k), tr = TR && bit(trunc, k), ed = bit(edge, k);
            const bool done = te || tr;
            const float cont = te ? 0.f : (tr ? d[1][k] : (ed ? B[k] : 0.f));
            al[k] = fmaf(P.gamma, cont, d[0][k]);
            be[k] = (done || ed) ? 0.f : P.gamma;
        }
    }
    template <int K, bool TR>
    __device__ static void finish(const Params&, const float (&)[kSlots][K], uint32_t, uint32_t,
                                  uint32_t, const float (&)[K], const float (&)[1],
                                  const float (&A)[K], float, float (&o0)[K], float (&)[K]) {
#pragma unroll
        for (int k = 0; k < K; ++k) o0[k] = A[k];
    }
};

// ---------------------------------------------------------------- forward scans (Sections 3.3.5-3.3.6)
// in: x. kDecay: eligibility traces (gamma lambda) vs. prefix sum (1). kStartsAt: a flag at t
// cuts the carry into t instead of into t+1.
template <bool kDecay, bool kStartsAt>
struct ForwardOp : OpBase {
    static constexpr bool kBackward = false;
    static constexpr int kSlots = 1;
    static constexpr int kTruncSlot = -1;
    static constexpr bool kFlags = true, kRowValue = false;
    static constexpr int kNbr = kStartsAt ? 0 : 1;  // done flag of the previous step
    static constexpr bool slot_used(int s, bool) { return s < 1; }

    template <int K>
    __device__ static void nbr_export(const Params&, const float (&)[kSlots][K], uint32_t done,
                                      float (&nb)[kNbr > 0 ? kNbr : 1]) {
        nb[0] = bit(done, K - 1) ? 1.f : 0.f;
    }
    // Raw flag bytes of the previous step (as 32-bit patterns); a missing flag array is read
    // from the data input instead (always in bounds) and ignored.
    static constexpr int kNbrRaw = 2;
    template <typename DT>
    __device__ static void nbr_load_raw(const Args& a, int64_t p, float (&raw)[kNbrRaw]) {
        const uint8_t* fallback = reinterpret_cast<const uint8_t*>(a.in[0]);
        raw[0] = __uint_as_float(uint32_t((a.term ? a.term : fallback)[p]));
        raw[1] = __uint_as_float(uint32_t((a.trunc ? a.trunc : fallback)[p]));
    }
    __device__ static void nbr_fix(const Args& a, const float (&raw)[kNbrRaw],
                                   float (&nb)[kNbr > 0 ? kNbr : 1]) {
        const bool t = a.term && __float_as_uint(raw[0]) != 0u;
        const bool r = a.trunc && __float_as_uint(raw[1]) != 0u;
        nb[0] = (t || r) ? 1.f : 0.f;
    }
    template <int K, bool TR>
    __device__ static void build(const Params& P, const float (&d)[kSlots][K], uint32_t term,
                                 uint32_t trunc, uint32_t edge, const float (&)[K],
                                 const float (&nb)[kNbr > 0 ? kNbr : 1], float (&al)[K],
                                 float (&be)[K]) {
        const float decay = kDecay ? P.gamma * P.lambda : 1.f;
        const uint32_t done = term | (TR ? trunc : 0u);
#pragma unroll
        for (int k = 0; k < K; ++k) {
            bool cut;
            if (kStartsAt) cut = bit(done, k);
            else cut = (k > 0) ? bit(done, k - 1) : (nb[0] != 0.f);
            al[k] = d[0][k];
            be[k] = (cut || bit(edge, k)) ? 0.f : decay;
        }
    }
    template <int K, bool TR>
    __device__ static void finish(const Params&, const float (&)[kSlots][K], uint32_t, uint32_t,
                                  uint32_t, const float (&)[K], const float (&)[kNbr > 0 ? kNbr : 1],
                                  const float (&A)[K], float, float (&o0)[K], float (&)[K]) {
#pragma unroll
        for (int k = 0; k < K; ++k) o0[k] = A[k];
    }
};

// ---------------------------------------------------------------- bare recurrence (Section 4.1)
// in: alpha, beta; the per-row carry enters at the row edge.
template <bool kBack>
struct AffineOp : OpBase {
    static constexpr bool kBackward = kBack;
    static constexpr int kSlots = 2;
    static constexpr int kTruncSlot = -1;
    static constexpr bool kFlags = false, kRowValue = true;
    static constexpr int kNbr = 0;
    static constexpr bool slot_used(int s, bool) { return s < 2; }

    template <int K>
    __device__ static void nbr_export(const Params&, const float (&)[kSlots][K], uint32_t, float (&)[1]) {}
    static constexpr int kNbrRaw = 1;
    template <typename DT>
    __device__ static void nbr_load_raw(const Args&, int64_t, float (&)[1]) {}
    __device__ static void nbr_fix(const Args&, const float (&)[1], float (&)[1]) {}
    template <int K, bool TR>
    __device__ static void build(const Params&, const float (&d)[kSlots][K], uint32_t, uint32_t,
                                 uint32_t edge, const float (&B)[K], const float (&)[1],
                                 float (&al)[K], float (&be)[K]) {
#pragma unroll
        for (int k = 0; k < K; ++k) {
            const bool ed = bit(edge, k);
            al[k] = ed ? fmaf(d[1][k], B[k], d[0][k]) : d[0][k];
            be[k] = ed ? 0.f : d[1][k];
        }
    }
    template <int K, bool TR>
    __device__ static void finish(const Params&, const float (&)[kSlots][K], uint32_t, uint32_t,
                                  uint32_t, const float (&)[K], const float (&)[1],
                                  const float (&A)[K], float, float (&o0)[K], float (&)[K]) {
#pragma unroll
        for (int k = 0; k < K; ++k) o0[k] = A[k];
    }
};

}  // namespace rlcs
