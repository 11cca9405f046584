// Device building blocks shared by every rlcs kernel: the affine pair and its composition
// (Eq. 2), the wave64 scan over lanes, and vectorised loads/stores of K consecutive elements.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace rlcs {

constexpr int kWave = 64;

// An affine map X -> a + b * X. Composing the maps of consecutive steps is the combine of
// Eq. 2: the step nearer to the output position is `outer`, the one nearer to the carry
// source (later in time for backward scans, earlier for forward scans) is `inner`.
struct Pair {
    float a, b;
};

__device__ __forceinline__ Pair identity_pair() { return Pair{0.f, 1.f}; }

__device__ __forceinline__ Pair compose(Pair outer, Pair inner) {
    return Pair{fmaf(outer.b, inner.a, outer.a), outer.b * inner.b};
}

// Value of the map at X.
__device__ __forceinline__ float apply(Pair m, float x) { return fmaf(m.b, x, m.a); }

// Inclusive scan of lane aggregates across the wave, towards the carry source: for a backward
// scan lane l ends with lanes l..63 composed (suffix), for a forward scan lanes 0..l (prefix).
// log2(64) = 6 shuffle steps (Hillis-Steele, as traced in Appendix A).
template <bool kBackward>
__device__ __forceinline__ Pair wave_scan_inclusive(Pair v, int lane) {
#pragma unroll
    for (int s = 1; s < kWave; s <<= 1) {
        const float a = kBackward ? __shfl_down(v.a, s) : __shfl_up(v.a, s);
        const float b = kBackward ? __shfl_down(v.b, s) : __shfl_up(v.b, s);
        const bool has = kBackward ? (lane + s < kWave) : (lane >= s);
        if (has) v = compose(v, Pair{a, b});
    }
    return v;
}

// The inclusive value of the neighbouring lane on the carry-source side (identity at the wave
// edge): the composition of every lane strictly between this lane and the wave's edge.
template <bool kBackward>
__device__ __forceinline__ Pair wave_exclusive_from_inclusive(Pair incl, int lane) {
    const float a = kBackward ? __shfl_down(incl.a, 1) : __shfl_up(incl.a, 1);
    const float b = kBackward ? __shfl_down(incl.b, 1) : __shfl_up(incl.b, 1);
    const bool edge = kBackward ? (lane == kWave - 1) : (lane == 0);
    return edge ? identity_pair() : Pair{a, b};
}

// ------------------------------------------------------------------ element loads / stores

// Element types of floating inputs: float, or bfloat16 held as its 16-bit pattern.
struct bf16_t {
    uint16_t bits;
};

__device__ __forceinline__ float widen(float x) { return x; }
__device__ __forceinline__ float widen(bf16_t x) { return __uint_as_float(uint32_t(x.bits) << 16); }

template <typename DT>
__device__ __forceinline__ float load_one(const void* base, int64_t i) {
    return widen(reinterpret_cast<const DT*>(base)[i]);
}

// Raw 32-bit words -> K widened values.
template <typename DT, int K>
__device__ __forceinline__ void unpack_words(const uint32_t* w, float (&out)[K]) {
    if constexpr (sizeof(DT) == 4) {
#pragma unroll
        for (int k = 0; k < K; ++k) out[k] = __uint_as_float(w[k]);
    } else {
#pragma unroll
        for (int k = 0; k < K; ++k) {
            const uint32_t word = w[k >> 1];
            out[k] = __uint_as_float((k & 1) ? (word & 0xffff0000u) : (word << 16));
        }
    }
}

// K consecutive elements starting at p0 (a multiple of K). `full`: all K are in range and the
// pointer is 16-byte aligned, so the load is one or more 16-byte vector loads. Otherwise only
// elements whose bit is set in `valid` are read; the rest are 0.
template <typename DT, int K>
__device__ __forceinline__ void load_k(const void* base, int64_t p0, uint32_t valid, bool full,
                                       float (&out)[K]) {
    constexpr int kBytes = K * int(sizeof(DT));
    static_assert(kBytes % 16 == 0 || kBytes == 8, "vector width");
    if (full) {
        uint32_t w[kBytes / 4];
        const char* p = reinterpret_cast<const char*>(base) + p0 * int64_t(sizeof(DT));
        if constexpr (kBytes % 16 == 0) {
#pragma unroll
            for (int i = 0; i < kBytes / 16; ++i) {
                const uint4 u = reinterpret_cast<const uint4*>(p)[i];
                w[4 * i + 0] = u.x; w[4 * i + 1] = u.y; w[4 * i + 2] = u.z; w[4 * i + 3] = u.w;
            }
        } else {
            const uint2 u = *reinterpret_cast<const uint2*>(p);
            w[0] = u.x; w[1] = u.y;
        }
        unpack_words<DT, K>(w, out);
    } else {
#pragma unroll
        for (int k = 0; k < K; ++k)
            out[k] = ((valid >> k) & 1u) ? load_one<DT>(base, p0 + k) : 0.f;
    }
}

// Flags of K consecutive steps as a K-bit mask (bit k set: byte k nonzero).
template <int K>
__device__ __forceinline__ uint32_t load_flags_k(const uint8_t* base, int64_t p0, uint32_t valid,
                                                 bool full) {
    uint32_t m = 0;
    if (full) {
        uint32_t w[(K + 3) / 4];
        if constexpr (K == 4) {
            w[0] = *reinterpret_cast<const uint32_t*>(base + p0);
        } else if constexpr (K == 8) {
            const uint2 u = *reinterpret_cast<const uint2*>(base + p0);
            w[0] = u.x; w[1] = u.y;
        } else {
            static_assert(K == 16, "flag vector width");
            const uint4 u = *reinterpret_cast<const uint4*>(base + p0);
            w[0] = u.x; w[1] = u.y; w[2] = u.z; w[3] = u.w;
        }
#pragma unroll
        for (int k = 0; k < K; ++k) m |= (((w[k >> 2] >> (8 * (k & 3))) & 0xffu) != 0u) ? (1u << k) : 0u;
    } else {
#pragma unroll
        for (int k = 0; k < K; ++k)
            if ((valid >> k) & 1u) m |= (base[p0 + k] != 0) ? (1u << k) : 0u;
    }
    return m;
}

template <int K>
__device__ __forceinline__ void store_k(float* base, int64_t p0, uint32_t valid, bool full,
                                        const float (&v)[K]) {
    if (full) {
        float4* p = reinterpret_cast<float4*>(base + p0);
#pragma unroll
        for (int i = 0; i < K / 4; ++i) p[i] = make_float4(v[4 * i], v[4 * i + 1], v[4 * i + 2], v[4 * i + 3]);
    } else {
#pragma unroll
        for (int k = 0; k < K; ++k)
            if ((valid >> k) & 1u) base[p0 + k] = v[k];
    }
}

}  // namespace rlcs
